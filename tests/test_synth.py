"""The seeded input generators: determinism, layout and the workload distributions."""
import numpy as np
import pytest

import synth


def test_weights_are_deterministic_and_seeded():
    m = synth.small_model()
    a, b = synth.make_weights(m, seed=3), synth.make_weights(m, seed=3)
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, synth.make_weights(m, seed=4))
    assert a.dtype == np.float32 and a.size == synth.blob_size(m)


def test_layout_roundtrip_and_init_kinds():
    m = synth.small_model(d_model=32, n_heads=2, n_enc=4, n_dec=1, vocab=50)
    blob = synth.make_weights(m)
    named = synth.unpack(m, blob)
    np.testing.assert_array_equal(synth.pack(m, named), blob)
    assert named["E"].shape == (50, 32)
    assert named["enc.0.W_qkv"].shape == (32, 96)
    assert named["dec.0.W_kv"].shape == (32, 64)
    for l in range(1, m.n_enc + 2):
        row = named[f"dlcl.{l}"]
        assert row.shape == (l,)
        assert abs(row.mean() - 1.0 / l) < 0.1
    assert abs(named["enc.1.ln2.gamma"].mean() - 1.0) < 0.05
    assert abs(named["enc.1.ln2.beta"].mean()) < 0.05


def test_eos_boost_scales_only_the_eos_row():
    m = synth.small_model()
    a = synth.make_weights(m)
    b = synth.make_weights(m, eos_boost=4.0)
    E_a, E_b = synth.unpack(m, a)["E"], synth.unpack(m, b)["E"]
    np.testing.assert_allclose(E_b[synth.EOS_ID], 4.0 * E_a[synth.EOS_ID], rtol=1e-6)
    mask = np.ones(len(E_a), bool)
    mask[synth.EOS_ID] = False
    np.testing.assert_array_equal(E_a[mask], E_b[mask])


def test_tiny_sentences():
    w = synth.WORKLOADS["tiny"]
    ids, offs = synth.make_sentences(w.data, w.model.vocab)
    lens = np.diff(offs)
    assert len(lens) == 8 and lens.min() >= 8 and lens.max() <= 16
    assert ids.min() >= synth.FIRST_WORD_ID and ids.max() < w.model.vocab
    ids2, offs2 = synth.make_sentences(w.data, w.model.vocab)
    np.testing.assert_array_equal(ids, ids2)


@pytest.mark.parametrize("name,mean,mx", [("base-6-6", 25, 100), ("wide-30-6", 30, 200)])
def test_lognormal_lengths_and_zipf_ids(name, mean, mx):
    w = synth.WORKLOADS[name]
    ids, offs = synth.make_sentences(w.data, w.model.vocab)
    lens = np.diff(offs)
    assert lens.min() >= 1 and lens.max() <= mx
    assert abs(lens.mean() - mean) < 1.5
    assert ids.min() >= synth.FIRST_WORD_ID and ids.max() < w.model.vocab
    # Zipf(1.1): rank 1 (ID 4) is the most frequent and frequencies fall with rank
    counts = np.bincount(ids, minlength=w.model.vocab)
    assert counts[4] > counts[5] > counts[20] > counts[1000]
    ratio = counts[4] / counts[5]
    assert 1.6 < ratio < 2.7          # 2^1.1 = 2.14


def test_max_target_len_and_subset():
    s = synth.SearchSetup(max_len_a=1.5, max_len_b=10)
    assert synth.max_target_len(s, 25) == 47
    assert synth.max_target_len(s, 1) == 11
    assert synth.max_target_len(synth.WORKLOADS["tiny"].search, 13) == 24
    offs = np.array([0, 3, 10, 12, 20, 21], dtype=np.int64)
    sub = synth.stratified_subset(offs, 2)
    assert list(sub) == [3, 0]     # sorted by (-len, idx): 3 (8), 1 (7), 0 (3), 2 (2), 4 (1)
