"""Mutation check of the oracle's pins (CPU only; run as a script, not collected by pytest).

Each entry plants one plausible mistake in a temporary copy of oracle/prcr_oracle.py
(a dropped term, a wrong sign or index, a swapped operand, an off-by-one bound) and
runs the oracle test files against the copy; a pin must fail for every mistake.
The unmutated copy runs first and must pass.

    python tests/oracle_mutations.py
"""
import os
import shutil
import subprocess
import sys
import tempfile

SRC = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MUTS = [
 ("baseline", "", ""),
 ("sign flip lo", "np.concatenate([lo * c - hi * s", "np.concatenate([lo * c + hi * s"),
 ("sign flip hi", "hi * c + lo * s]", "hi * c - lo * s]"),
 ("swap partners", "np.concatenate([lo * c - hi * s, hi * c + lo * s]", "np.concatenate([hi * c - lo * s, lo * c + hi * s]"),
 ("invf index", "(-(2.0 * i) / head_dim)", "(-(2.0 * (i + 1)) / head_dim)"),
 ("invf exponent", "(-(2.0 * i) / head_dim)", "(-(1.0 * i) / head_dim)"),
 ("interleave h/w", "if i % 3 == 1 and i < 3 * s_h", "if i % 3 == 2 and i < 3 * s_h"),
 ("interleave cap", "i < 3 * s_w", "i < 3 * s_h"),
 ("section bound", "elif i < s_t + s_h:", "elif i < s_t + s_w + 1:"),
 ("pcr K-1", "(1 + (K - 1) * u)", "(1 + K * u)"),
 ("pcr L+1", "(L + 1) * (1 + (K - 1) * u)", "L * (1 + (K - 1) * u)"),
 ("pcr K+1", "/ Fraction(K + 1)", "/ Fraction(K)"),
 ("pcr anchor", "start = p_txt + 1 if mode == \"pcr_right\" else p_txt - L", "start = p_txt + 1 if mode == \"pcr_right\" else p_txt - L + 1"),
 ("pcr right anchor", "start = p_txt + 1 if mode == \"pcr_right\" else p_txt - L", "start = p_txt if mode == \"pcr_right\" else p_txt - L"),
 ("R2 midpoint", "u = Fraction(1, 2)", "u = Fraction(0)"),
 ("u denom", "Fraction(int(c[j, a]) - lo[a], hi[a] - lo[a])", "Fraction(int(c[j, a]) - lo[a], hi[a] - lo[a] + 1)"),
 ("shift start", "v = (p_txt + 1) + (int(c[j, a]) - lo[a])", "v = p_txt + (int(c[j, a]) - lo[a])"),
 ("shift next", "(p_txt + 1 if top is None else top + 1)", "(p_txt + 1 if top is None else top)"),
 ("lpa", "out[j] = float(p_txt + j + 1)", "out[j] = float(p_txt + j)"),
 ("uir", "Fraction(j + 1, K + 1)", "Fraction(j, K + 1)"),
 ("bf16 floor", "np.rint(np.ldexp(y, -q))", "np.floor(np.ldexp(y, -q))"),
 ("bf16 precision", "q = np.maximum(e - 8, -133)", "q = np.maximum(e - 9, -133)"),
 ("bf16 subnormal", "q = np.maximum(e - 8, -133)", "q = np.maximum(e - 8, -126)"),
 ("slot +1", "slot, where = slot_of(cache, b, int(cache_len[b]) + j)", "slot, where = slot_of(cache, b, int(cache_len[b]) + j + 1)"),
 ("paged off", "return blk * bs + s % bs, (blk, s % bs)", "return blk * bs + s % bs, (blk, (s + 1) % bs)"),
 ("paged lb", "lb = s // bs", "lb = (s + 1) // bs"),
 ("contig slot id", "return b * cache[\"s_max\"] + s, (b, s)", "return b * cache[\"s_max\"] + s + 1, (b, s)"),
 ("newlen", "new_len[b] = int(cache_len[b]) + (s1 - s0)", "new_len[b] = int(cache_len[b])"),
 ("value from K", "vv = mem[\"v\"][b, m]", "vv = mem[\"k\"][b, m]"),
 ("store layer", "mem_k[b, m, layer] = raw_k[b, r]", "mem_k[b, m, 0] = raw_k[b, r]"),
 ("index check", "if m < 0 or m >= int(mem[\"n_visual\"][b]):", "if m < 0 or m > int(mem[\"n_visual\"][b]):"),
 ("block check", "if blk < 0 or blk >= cache[\"n_blocks\"]:", "if blk < 0 or blk > cache[\"n_blocks\"]:"),
 ("konly slot bound", "if vsl < 0 or vsl >= int(cache_len[b]):", "if vsl < 0 or vsl > int(cache_len[b]):"),
 ("konly paged src k", "vv = np.array(cache[\"v\"][:, src_where[0], src_where[1]], copy=True)", "vv = np.array(cache[\"k\"][:, src_where[0], src_where[1]], copy=True)"),
 ("konly contig src", "vv = np.array(cache[\"v\"][b, :, :, src_where[1]], copy=True)", "vv = np.array(cache[\"v\"][b, :, :, vsl - 1], copy=True)"),
 ("prefill v_slot", "vs[b, m] = int(cache_start[b]) + s if slot is not None else -1", "vs[b, m] = int(cache_start[b]) + s + 1 if slot is not None else -1"),
 ("store v skip", "            if mem_v is not None:\n                mem_v[b, m, layer] = raw_v[b, r]", "            if False:\n                mem_v[b, m, layer] = raw_v[b, r]"),
 ("decode norm", "out[b, qh] = (w / w.sum()) @ V", "out[b, qh] = w @ V"),
 ("decode gqa", "qh = kvh * G + g", "qh = g * n_kv + kvh"),
 ("decode qpos", "p = np.full(3, float(q_pos[b]))", "p = np.full(3, float(q_pos[b]) + 1)"),
 ("decode scale", "s = (K @ qr) * scale", "s = (K @ qr) * scale * 2"),
 ("decode empty", "        if n == 0:\n            continue", "        if n <= 1:\n            continue"),
]


def run(name, a, b):
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    try:
        for x in ("oracle", "tests"):
            shutil.copytree(os.path.join(SRC, x), os.path.join(d, x),
                            ignore=shutil.ignore_patterns("__pycache__"))
        for f in ("pytest.ini", "workloads.py"):
            shutil.copy(os.path.join(SRC, f), d)
        p = os.path.join(d, "oracle", "prcr_oracle.py")
        text = open(p).read()
        if a:
            if a not in text:
                return "PATTERN NOT FOUND"
            open(p, "w").write(text.replace(a, b, 1))
        files = sorted(os.path.join("tests", f) for f in os.listdir(os.path.join(d, "tests"))
                       if f.startswith("test_oracle_"))
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            *files], cwd=d, capture_output=True, text=True)
        if r.returncode == 0:
            return "passes"
        first = [l for l in r.stdout.splitlines() if l.startswith("FAILED") or "Error" in l][:1]
        return "caught " + (first[0][:90] if first else "")
    finally:
        shutil.rmtree(d, ignore_errors=True)


def main():
    bad = 0
    for name, a, b in MUTS:
        res = run(name, a, b)
        ok = res == "passes" if name == "baseline" else res.startswith("caught")
        bad += not ok
        print(f"{name:20s} {res}", flush=True)
    print("all mistakes caught" if bad == 0 else f"{bad} entries not as expected")
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())
