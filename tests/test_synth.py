"""kf_synth: the seeded input generators shared by both sides (no method arithmetic)."""
import os

import numpy as np

import kf_synth as S

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _kat():
    rows = []
    for line in open(os.path.join(GOLD, "philox4x32_10_kat.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[:4], w[4:6], w[6:10]))
    return rows


def test_philox_kat():
    for ctr, key, out in _kat():
        got = S.philox4x32_10(*[np.uint32(c) for c in ctr], key=tuple(key))
        assert [int(x) for x in got] == out


def test_noise_is_24bit_uniform():
    u = S.noise_block(7, 8, 0, 512)
    assert u.dtype == np.float32 and u.shape == (8, 512)
    assert (u >= 0).all() and (u < 1).all()
    assert np.all((u * 16777216.0) == np.round(u * 16777216.0))
    assert abs(float(u.mean()) - 0.5) < 0.02


def test_noise_indexed_by_position():
    a = S.noise_block(3, 4, 10, 8)
    b = S.noise_block(3, 4, 14, 4)
    np.testing.assert_array_equal(a[:, 4:], b)


def test_normal_moments():
    x = S.normal(0, 5, 400_000, 0.02)
    assert abs(float(x.std()) - 0.02) < 2e-4
    assert abs(float(x.mean())) < 2e-4


def test_prompts_in_range():
    z = S.prompts_zipf(1, 16, 128, 50257)
    assert z.min() >= 0 and z.max() < 50257
    # Zipf(1.1): rank 1 is the most frequent id
    assert np.bincount(z.reshape(-1)).argmax() == 0
    u = S.prompts_uniform(1, 4, 16, 1024)
    assert u.min() >= 0 and u.max() < 1024


def test_blob_layout_and_sizes():
    cfg = S.WORKLOADS["toy"]["cfg"]
    w = S.make_weights(cfg, seed=0)
    blob = S.pack_blob(cfg, w)
    assert blob.size == 16 + S.n_params(cfg)
    hdr = blob[:16].view(np.int32)
    assert hdr[0] == S.BLOB_MAGIC and list(hdr[2:9]) == [2, 128, 4, 512, 1024, 128, 0]
    assert np.all(w["l0.b_qkv"] == 0) and np.all(w["lnf_g"] == 1)
    w2 = S.make_weights(cfg, seed=0, random_affine=True)
    assert np.any(w2["l0.b_qkv"] != 0) and np.any(w2["lnf_g"] != 1)
    np.testing.assert_array_equal(w["tok_emb"], w2["tok_emb"])
