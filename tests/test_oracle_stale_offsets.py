"""Why the revisited tokens get new positions (Sec. 3.2, Eq. (5), Table 2), shown on
synthetic scores with no model.

Direct reuse (IDENTITY) keeps a revisited key at its original coordinates, so a
query decoded at p_next sees it p_next - c positions in the past on every axis;
rotary scores depend only on that offset (Eq. (5)).  PCR puts every revisited
token within L + 1 positions of the query.  The tests check the offsets, the
closed-form rotary score of an aligned query and key at those offsets, and the
attention mass a decoding query puts on the evidence it looks for, through the
oracle's decode attention (Eq. (14)), among recent text keys.

Shape: a 36 x 36 image whose prompt offset is 100, a 12 x 12 revisited region,
p_txt = 1599, L = 2, head_dim 128, sections [16, 24, 24], theta 1e6.
"""
import numpy as np

import oracle

D, SECTIONS, THETA, L = 128, (16, 24, 24), 1e6, 2
ROPE = {"head_dim": D, "sections": SECTIONS, "interleaved": False, "theta": THETA}
Q0, GRID, P_TXT = 100, 36, 1599
COORDS = np.array([(Q0, Q0 + h, Q0 + w) for h in range(GRID) for w in range(GRID)])
SEL = np.array([h * GRID + w for h in range(10, 22) for w in range(5, 17)])


def _aligned_score(offsets):
    """<R(p_next) x, R(p) x> / |x|^2 for a key whose rotary pairs all have the same
    norm: the mean over pairs of cos(offset on the pair's axis * inv_freq), Eq. (5)."""
    invf = oracle.inv_freq(THETA, D)
    axis = oracle.pair_axis(D, SECTIONS, False)
    return np.cos(offsets[:, axis] * invf).mean(axis=1)


def test_offsets_pcr_local_identity_stale():
    pcr, nxt = oracle.reassign(COORDS[SEL], P_TXT, "pcr", L)
    ident, nxt_i = oracle.reassign(COORDS[SEL], P_TXT, "identity", L)
    assert nxt == nxt_i == P_TXT + 1
    off_pcr, off_id = nxt - pcr, nxt - ident
    assert (off_pcr > 0).all() and (off_pcr < L + 1).all()
    assert off_id.min() == P_TXT + 1 - (Q0 + 21) and off_id.max() == P_TXT + 1 - Q0


def test_aligned_rotary_score_closed_form_and_decay():
    rng = np.random.default_rng(7)
    invf = oracle.inv_freq(THETA, D)
    axis = oracle.pair_axis(D, SECTIONS, False)
    scores = {}
    for mode in ("pcr", "identity"):
        pos, nxt = oracle.reassign(COORDS[SEL], P_TXT, mode, L)
        # the rotated score of a random key with itself equals the closed form
        # weighted by its own pair norms
        x = rng.standard_normal((len(SEL), D))
        got = (oracle.rotate_keys(x, pos, invf, axis) *
               oracle.rotate_keys(x, np.full_like(pos, float(nxt)), invf, axis)).sum(1)
        norm2 = x[:, :D // 2] ** 2 + x[:, D // 2:] ** 2
        want = (norm2 * np.cos((nxt - pos)[:, axis] * invf)).sum(1)
        assert np.allclose(got, want, rtol=0, atol=1e-10)
        scores[mode] = _aligned_score(nxt - pos)
    # PCR keeps an aligned score near its zero-offset value 1; direct reuse loses
    # most of it to the stale offsets
    assert scores["pcr"].min() > 0.85
    assert scores["identity"].mean() < 0.5
    assert (scores["pcr"] > scores["identity"]).all()


def test_attention_mass_on_revisited_evidence():
    """A query that looks for one revisited token (q = half its raw key), decoded
    at p_next over 256 recent text keys plus the 144 revisited keys: the value rows
    are indicators, so the oracle's attention output reads off the mass on that
    token."""
    rng = np.random.default_rng(11)
    invf = oracle.inv_freq(THETA, D)
    axis = oracle.pair_axis(D, SECTIONS, False)
    K, n_txt = len(SEL), 256
    k_vis = rng.standard_normal((K, D))
    k_txt = rng.standard_normal((n_txt, D))
    p_t = np.arange(P_TXT - n_txt + 1, P_TXT + 1, dtype=np.float64)
    kt = oracle.rotate_keys(k_txt, np.repeat(p_t[:, None], 3, 1), invf, axis)
    picks = np.arange(0, K, 7)
    mass = {}
    for mode in ("pcr", "identity"):
        pos, nxt = oracle.reassign(COORDS[SEL], P_TXT, mode, L)
        keys = np.concatenate([kt, oracle.rotate_keys(k_vis, pos, invf, axis)])
        n = len(keys)
        vals = np.zeros((n, D))
        vals[n_txt + picks, np.arange(len(picks))] = 1.0     # one indicator column per pick
        cache = {"paged": False, "s_max": n, "k": keys[None, None, None].astype(np.float32),
                 "v": vals[None, None, None].astype(np.float32)}
        out = []
        for c, j in enumerate(picks):
            o = oracle.decode_attention(ROPE, cache, 0, (0.5 * k_vis[j])[None, None].astype(np.float32),
                                        np.array([nxt]), np.array([n]), D ** -0.5, "f32")
            out.append(o[0, 0, c])
        mass[mode] = np.array(out)
    assert (mass["pcr"] > mass["identity"]).all()
    assert mass["pcr"].mean() > 5 * mass["identity"].mean()
