"""Pins of the m-bit sign-magnitude quantizer of Appendix A (the paper's
experimental compressor with Hou et al.'s infinity-norm scale)."""
import numpy as np
import pytest

from conftest import load_golden


@pytest.mark.parametrize("m", [4, 8])
def test_code_layout_on_exact_grid(oracle_mod, m):
    g = load_golden("mbit_code_example.txt")
    v = np.array(g["m%d_v" % m], np.float32)
    k = (1 << (m - 1)) - 1
    sigma = oracle_mod.scale(v, "linf")
    assert sigma == np.float32(g["m%d_scale" % m][0])
    for t in range(20):
        bits, lv, phat, e = oracle_mod.qsgd_encode(v, sigma, k, 5, 0, t)
        np.testing.assert_array_equal(phat, v)
        codes = oracle_mod.mbit_fields(bits, lv, m)
        np.testing.assert_array_equal(codes, np.array(g["m%d_codes" % m], np.uint16))
        word = oracle_mod.pack_bits(codes, m, 1)
        assert int(word[0]) == int(g["m%d_word" % m][0], 16)


@pytest.mark.parametrize("m", [4, 8])
def test_fields_roundtrip(oracle_mod, m):
    rng = np.random.default_rng(m)
    k = (1 << (m - 1)) - 1
    bits = rng.integers(0, 2, 5000).astype(np.uint8)
    lv = rng.integers(0, k + 1, 5000).astype(np.uint16)
    f = oracle_mod.mbit_fields(bits, lv, m)
    assert f.max() < (1 << m)
    sg, lv2 = oracle_mod.mbit_split(f, m)
    np.testing.assert_array_equal(sg, bits)
    np.testing.assert_array_equal(lv2, lv)


@pytest.mark.parametrize("m", [4, 8])
def test_mbit_step_decodes_to_the_quantized_vector(oracle_mod, m):
    """One iteration with the m-bit compressor: the server's decode of the
    packed codes equals the workers' p-hat (e + p-hat reproduces p), and the
    code plane holds sign and level in the stated bits."""
    import synth
    from synth.configs import custom
    w = custom(d=3000, M=3, kind="mbit", levels=m, norm="linf", seg_offsets=[0, 1000, 3000], eta=1e-2, seed=3)
    cfg = w.as_dict()
    G = synth.gradients_np(w, 1)
    E = np.zeros((w.M, w.ld), np.float32)
    W = synth.init_params_np(w)
    P = np.stack([oracle_mod.ef_accumulate(np.float32(w.eta), G[r, :w.d], E[r, :w.d]) for r in range(w.M)])
    out = oracle_mod.step(cfg, np.float32(w.eta), 1, G, E, W)
    k = (1 << (m - 1)) - 1
    for r in range(w.M):
        codes = oracle_mod.unpack_bits(out["level"][r], m, w.d)
        sg, lv = oracle_mod.mbit_split(codes, m)
        np.testing.assert_array_equal(sg, np.signbit(P[r]).astype(np.uint16))
        assert lv.max() <= k
        for j, (a, b) in enumerate(zip(cfg["seg_offsets"][:-1], cfg["seg_offsets"][1:])):
            assert out["scale"][r, j] == np.abs(P[r, a:b]).max()
            ph = oracle_mod.decode_segment("qsgd", sg[a:b], lv[a:b], out["scale"][r, j], k)
            back = (E[r, a:b] + ph).astype(np.float32)
            assert np.all(np.abs(back - P[r, a:b]) <= np.spacing(np.maximum(np.abs(P[r, a:b]), np.abs(ph))))
