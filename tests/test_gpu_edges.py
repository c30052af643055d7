"""GPU edge cases of nt_translate: input it must reject (an empty sentence, a source past
the position table, a token ID outside the vocabulary, a target limit past the position
table), a model that keeps working after a rejected call, the longest source the
position table allows, one-step target limits, and source lengths at the edges of the
decoder cross-attention's key blocks and chunks.  Parity is against the oracle in
fp32 (token IDs under the near-tie protocol, teacher-forced logits within 1e-3)."""
import numpy as np
import pytest

import oracle
import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = synth.ModelShape(64, 2, 256, 2, 1, 101)


def _csr(sents):
    ids = np.concatenate([np.asarray(s, dtype=np.int32) for s in sents])
    offs = np.concatenate([[0], np.cumsum([len(s) for s in sents])]).astype(np.int64)
    return ids, offs


def test_invalid_inputs_are_rejected_and_the_model_stays_usable():
    from paper_2109_08008_amd import nt
    blob = synth.make_weights(SHAPE, seed=71, lively=True)
    model = G.new_model(SHAPE, blob, "f32")
    search = synth.SearchSetup(beam=1, max_len_a=1.0, max_len_b=4)
    P = synth.MAX_POSITIONS
    cases = {
        "empty sentence": ([[5, 6], [], [7]], search),
        "source past the position table": ([[5] * (P + 1)], search),
        "token id = vocab": ([[5, SHAPE.vocab, 7]], search),
        "negative token id": ([[5, -1]], search),
        "target limit past the position table": ([[5] * 600], synth.replace(search, max_len_a=2.0, max_len_b=0)),
    }
    for name, (sents, s) in cases.items():
        ids, offs = _csr(sents)
        with pytest.raises(nt.NTError) as err:
            model.translate(ids, offs, s)
        assert err.value.status == nt.NT_E_INVALID, (name, err.value)
    srcs = [[5, 6, 7, 8], [9], [10, 11, 12]]
    ids, offs = _csr(srcs)
    toks, scores, _ = model.translate(ids, offs, search)
    om = G.oracle_model(SHAPE, blob, "f32")
    ties = sum(G.compare_greedy_ids(om, s, tk, synth.max_target_len(search, len(s))) for s, tk in zip(srcs, toks))
    assert ties <= 1
    model.close()


def test_longest_source_the_position_table_allows():
    blob = synth.make_weights(SHAPE, seed=72, lively=True)
    rng = np.random.default_rng(73)
    P = synth.MAX_POSITIONS
    srcs = [list(rng.integers(3, SHAPE.vocab, size=P)), [4], list(rng.integers(3, SHAPE.vocab, size=P - 1))]
    tgts = [list(rng.integers(3, SHAPE.vocab, size=3)) for _ in srcs]
    model = G.new_model(SHAPE, blob, "f32")
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, SHAPE.vocab)
    om = G.oracle_model(SHAPE, blob, "f32")
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        np.testing.assert_allclose(got[b], om.teacher_forced_logits(s, tg), atol=1e-3)
    # and translated with greedy search
    search = synth.SearchSetup(beam=1, max_len_a=0.0, max_len_b=6)
    ids, offs = _csr(srcs)
    toks, _, _ = model.translate(ids, offs, search)
    ties = sum(G.compare_greedy_ids(om, s, tk, 6) for s, tk in zip(srcs, toks))
    assert ties <= 1
    model.close()


@pytest.mark.parametrize("beam", [1, 4])
def test_one_step_target_limit(beam):
    """max target length 1: every hypothesis ends after one step (EOS or the limit)."""
    blob = synth.make_weights(SHAPE, seed=74, lively=True)
    srcs = [[5, 6, 7], [8], [9, 10]]
    ids, offs = _csr(srcs)
    search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=0.0, max_len_b=1)
    model = G.new_model(SHAPE, blob, "f32")
    toks, scores, _ = model.translate(ids, offs, search)
    om = G.oracle_model(SHAPE, blob, "f32")
    for s, tk, sc in zip(srcs, toks, scores):
        assert len(tk) <= 1
        if beam > 1:
            ref = oracle.translate(om, s, search)
            assert list(tk) == list(ref.tokens)
            assert abs(sc - ref.score) <= 1e-3
        else:
            assert G.compare_greedy_ids(om, s, tk, 1) <= 1
    model.close()


def test_undersized_workspace_is_reported():
    """NT_E_WORKSPACE from nt_encode and nt_translate when the workspace is one 256-byte
    granule short, with the required size in the message; at the stated size both run."""
    from paper_2109_08008_amd import nt
    torch = G.torch_cuda()
    blob = synth.make_weights(SHAPE, seed=75, lively=True)
    model = G.new_model(SHAPE, blob, "f32")
    srcs = [[5, 6, 7], [8], [9, 10]]
    search = synth.SearchSetup(beam=2, max_len_a=1.0, max_len_b=3)
    sc = nt.search_cfg(search)
    arr, lens = G.pad_batch(srcs)
    B, S = arr.shape
    need = nt.nt_workspace_size(model.handle, sc, B, S)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    d_src, d_len = torch.from_numpy(arr).cuda(), torch.from_numpy(lens).cuda()
    with pytest.raises(nt.NTError) as err:
        nt.nt_encode(model.handle, d_src.data_ptr(), d_len.data_ptr(), lens, B, S, sc, ws.data_ptr(), need - 256)
    assert err.value.status == nt.NT_E_WORKSPACE and str(need) in err.value.message, err.value
    st = nt.nt_encode(model.handle, d_src.data_ptr(), d_len.data_ptr(), lens, B, S, sc, ws.data_ptr(), need)
    nt.nt_free_state(st)
    ids, offs = _csr(srcs)
    need_t = nt.nt_translate_workspace_size(model.handle, sc, offs)
    wst = torch.empty(need_t, dtype=torch.uint8, device="cuda")
    cap = sum(synth.max_target_len(search, len(s)) for s in srcs)
    with pytest.raises(nt.NTError) as err:
        nt.nt_translate(model.handle, sc, ids, offs, cap, wst.data_ptr(), need_t - 256)
    assert err.value.status == nt.NT_E_WORKSPACE and str(need_t) in err.value.message, err.value
    out, out_off, _, _ = nt.nt_translate(model.handle, sc, ids, offs, cap, wst.data_ptr(), need_t)
    assert out_off[-1] <= cap
    model.close()


def test_steps_after_the_end_and_early_reads_are_state_errors():
    """nt_dec_state_read before every sentence has finished and nt_decode_step after it
    give NT_E_STATE; the step-level results equal the oracle's beam search."""
    from paper_2109_08008_amd import nt
    blob = synth.make_weights(SHAPE, seed=76, lively=True)
    model = G.new_model(SHAPE, blob, "f32")
    srcs = [[5, 6, 7, 8], [9], [10, 11]]
    search = synth.SearchSetup(beam=2, len_penalty=0.6, max_len_a=1.0, max_len_b=3)
    st, keep = G.gpu_encode(model, srcs, search)
    try:
        with pytest.raises(nt.NTError) as err:
            nt.nt_dec_state_read(st)
        assert err.value.status == nt.NT_E_STATE, err.value
        limit = max(synth.max_target_len(search, len(s)) for s in srcs)
        steps = 0
        while nt.nt_decode_step(st) > 0:
            steps += 1
            assert steps <= limit
        for _ in range(2):
            with pytest.raises(nt.NTError) as err:
                nt.nt_decode_step(st)
            assert err.value.status == nt.NT_E_STATE, err.value
        toks, scores, _ = nt.nt_dec_state_read(st)
    finally:
        nt.nt_free_state(st)
    om = G.oracle_model(SHAPE, blob, "f32")
    for s, tk, sc in zip(srcs, toks, scores):
        ref = oracle.translate(om, s, search)
        assert list(tk) == list(ref.tokens)
        assert abs(sc - ref.score) <= 1e-3
    model.close()


def test_beam_wider_than_16_is_unsupported():
    from paper_2109_08008_amd import nt
    blob = synth.make_weights(SHAPE, seed=77)
    model = G.new_model(SHAPE, blob, "f32")
    wide = synth.SearchSetup(beam=17, max_len_a=1.0, max_len_b=3)
    ids, offs = _csr([[5, 6], [7]])
    with pytest.raises(nt.NTError) as err:
        nt.nt_workspace_size(model.handle, nt.search_cfg(wide), 2, 2)
    assert err.value.status == nt.NT_E_UNSUPPORTED, err.value
    with pytest.raises(nt.NTError) as err:
        model.translate(ids, offs, wide)
    assert err.value.status == nt.NT_E_UNSUPPORTED, err.value
    toks, _, _ = model.translate(ids, offs, synth.replace(wide, beam=16))   # the widest accepted
    assert all(len(t) <= 3 for t in toks)
    model.close()


@pytest.mark.parametrize("beam", [1, 4])
def test_target_length_cap(beam):
    """max_len_cap lowers every sentence's limit floor(a * len) + b to the cap (the
    paper caps targets at 200 tokens, Sec. 4.4); a negative cap is rejected."""
    from paper_2109_08008_amd import nt
    blob = synth.make_weights(SHAPE, seed=78, lively=True, eos_boost=1.0)
    rng = np.random.default_rng(79)
    srcs = [list(rng.integers(4, SHAPE.vocab, size=n)) for n in (12, 3, 7, 20)]
    ids, offs = _csr(srcs)
    search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=10, max_len_cap=5)
    model = G.new_model(SHAPE, blob, "f32")
    toks, scores, _ = model.translate(ids, offs, search)
    om = G.oracle_model(SHAPE, blob, "f32")
    for s, tk, sc in zip(srcs, toks, scores):
        assert synth.max_target_len(search, len(s)) == 5 and len(tk) <= 5
        if beam > 1:
            ref = oracle.translate(om, s, search)
            assert list(tk) == list(ref.tokens)
            assert abs(sc - ref.score) <= 1e-3
        else:
            assert G.compare_greedy_ids(om, s, tk, 5) <= 1
    with pytest.raises(nt.NTError) as err:
        model.translate(ids, offs, synth.replace(search, max_len_cap=-1))
    assert err.value.status == nt.NT_E_INVALID, err.value
    model.close()


def test_cross_attention_chunk_edges():
    """Source lengths at and next to the decoder cross-attention's 16-key blocks and
    64-key chunks, at d_head 64 (a chunk's key blocks past the source length re-read its
    last key and are masked): fp32 teacher-forced logits within 1e-3 of the oracle, and
    the per-token log-probs of beam-4 translations within 1e-3 of the oracle's logits on
    the same tokens."""
    shape = synth.ModelShape(128, 2, 256, 1, 1, 101)
    blob = synth.make_weights(shape, seed=77, lively=True, eos_boost=2.0)
    rng = np.random.default_rng(78)
    lengths = [1, 15, 16, 17, 31, 32, 33, 47, 48, 49, 63, 64, 65, 127, 128, 129]
    srcs = [list(rng.integers(3, shape.vocab, size=L)) for L in lengths]
    tgts = [list(rng.integers(3, shape.vocab, size=3)) for _ in srcs]
    model = G.new_model(shape, blob, "f32")
    om = G.oracle_model(shape, blob, "f32")
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        np.testing.assert_allclose(got[b], om.teacher_forced_logits(s, tg), atol=1e-3, err_msg=f"length {len(s)}")
    ids, offs = _csr(srcs)
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=0.0, max_len_b=4)
    toks, _, logp = model.translate(ids, offs, search)
    assert sum(len(t) for t in toks) > len(toks)
    for s, tk, lp in zip(srcs, toks, logp):
        ref = om.teacher_forced_logits(s, list(tk))
        lse = np.log(np.exp(ref - ref.max(1, keepdims=True)).sum(1)) + ref.max(1)
        want = np.array([ref[t, tk[t]] - lse[t] for t in range(len(tk))])
        np.testing.assert_allclose(np.asarray(lp), want, atol=1e-3, err_msg=f"length {len(s)}")
    model.close()


@pytest.mark.parametrize("beam", [1, 4])
def test_long_k_decoder_projection_is_batch_invariant(beam):
    """The decoder's K = 4096 projection (the second FFN GEMM at d_ff 4096, the longest
    k-loop of a step, on its four-stage tile): fp16 translations are bitwise the same
    whatever the batching, and the fp16 teacher-forced logits stay within 5e-2 of the
    oracle."""
    shape = synth.ModelShape(1024, 16, 4096, 1, 1, 101)
    blob = synth.make_weights(shape, seed=79, lively=True, eos_boost=4.0)
    ids, offs = synth.make_sentences(synth.DataSetup(24, "uniform", 1, 30, "uniform"), shape.vocab, seed=80)
    model = G.new_model(shape, blob, "f16")
    base = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=8192, prune=1)
    ref = model.translate(ids, offs, base)
    assert sum(len(t) for t in ref[0]) > len(ref[0])
    for kw in [dict(token_budget=64), dict(token_budget=0, max_batch_sents=1)]:
        t, s, _ = model.translate(ids, offs, synth.replace(base, **kw))
        for a, b in zip(ref[0], t):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(ref[1], s)
    srcs = synth.sentence_list(ids, offs)[:6]
    rng = np.random.default_rng(81)
    tgts = [list(rng.integers(3, shape.vocab, size=4)) for _ in srcs]
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, "f16")
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        assert float(np.abs(got[b] - om.teacher_forced_logits(s, tg)).max()) <= 5e-2, len(s)
    model.close()
