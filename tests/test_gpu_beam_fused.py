"""Beam selection without stored logits (the default) against the plain path that stores
the fp32 logits and scans every row (nt_set_beam_fused(0)).  Both select from the same
logit bits; only each row's log-sum-exp is summed in another order (merged from the
per-tile records, against one pass over the row), a few units in the last place.  So
token IDs must be identical, and scores and per-token log-probs equal within 1e-6
relative, at every beam width the library accepts, in every dtype, with vocabularies
that end in a ragged tile or hold fewer tiles than 2K, with and without pruning.  Step
by step, the logits a caller asks for are the same bits on both paths.  The plain path's selection is pinned against NumPy elsewhere
(test_gpu_select), and the search as a whole against the oracle (test_gpu_parity, which
runs the fused default)."""
import numpy as np
import pytest

import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu


def _translate(model, ids, offs, search, fused):
    from paper_2109_08008_amd import nt
    nt.nt_set_beam_fused(fused)
    try:
        return model.translate(ids, offs, search)
    finally:
        nt.nt_set_beam_fused(True)


CASES = [
    # (shape, dtype, beam, prune)
    (synth.ModelShape(64, 2, 256, 2, 1, 101), "f32", 2, 1),       # one tile, fewer than 2K at K >= 1
    (synth.ModelShape(64, 2, 256, 2, 1, 101), "f32", 16, 1),
    (synth.ModelShape(128, 4, 512, 2, 2, 517), "f16", 4, 1),      # five tiles, the last ragged
    (synth.ModelShape(128, 4, 512, 2, 2, 517), "bf16", 8, 0),
    (synth.ModelShape(256, 4, 1024, 2, 2, 2000), "f16", 3, 1),
    (synth.ModelShape(256, 4, 1024, 2, 2, 2000), "f32", 16, 0),   # 2K = 32 tiles of 16
]


@pytest.mark.parametrize("shape,dtype,beam,prune", CASES, ids=[f"V{c[0].vocab}-{c[1]}-K{c[2]}-p{c[3]}" for c in CASES])
def test_fused_beam_equals_the_plain_scan(shape, dtype, beam, prune):
    blob = synth.make_weights(shape, seed=91, lively=True, eos_boost=1.5)
    ids, offs = synth.make_sentences(synth.DataSetup(40, "uniform", 1, 24, "uniform"), shape.vocab, seed=92)
    search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.2, max_len_b=6, token_budget=256, prune=prune)
    model = G.new_model(shape, blob, dtype)
    fused = _translate(model, ids, offs, search, True)
    plain = _translate(model, ids, offs, search, False)
    model.close()
    assert sum(len(t) for t in fused[0]) > len(fused[0])   # hypotheses of varied length, not all empty
    for a, b in zip(fused[0], plain[0]):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(fused[1], plain[1], rtol=1e-6, atol=1e-6)
    for a, b in zip(fused[2], plain[2]):
        np.testing.assert_allclose(a, b, rtol=1e-6, atol=1e-6)


def test_logits_copy_out_is_the_same_on_both_paths():
    from paper_2109_08008_amd import nt
    torch = G.torch_cuda()
    shape = synth.ModelShape(128, 4, 512, 2, 2, 517)
    blob = synth.make_weights(shape, seed=93, lively=True, eos_boost=1.5)
    srcs = [[5, 6, 7, 8, 9], [10], [11, 12, 13], [14, 15]]
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.0, max_len_b=4, prune=1)
    model = G.new_model(shape, blob, "f16")
    runs = []
    for fused in (True, False):
        nt.nt_set_beam_fused(fused)
        try:
            st, keep = G.gpu_encode(model, srcs, search)
        finally:
            nt.nt_set_beam_fused(True)
        steps = []
        try:
            while True:
                buf = torch.full((len(srcs) * search.beam, shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
                alive = nt.nt_decode_step(st, 0, buf.data_ptr())
                steps.append(buf.cpu().numpy())
                if alive == 0:
                    break
            out = nt.nt_dec_state_read(st)
        finally:
            nt.nt_free_state(st)
        runs.append((steps, out))
    model.close()
    (fs, fo), (ps, po) = runs
    assert len(fs) == len(ps) and len(fs) >= 2
    for a, b in zip(fs, ps):
        np.testing.assert_array_equal(np.isnan(a), np.isnan(b))
        np.testing.assert_array_equal(np.nan_to_num(a), np.nan_to_num(b))
    for a, b in zip(fo[0], po[0]):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(fo[1], po[1], rtol=1e-6, atol=1e-6)


def test_fused_beam_with_more_pairs_than_the_sort_holds_in_lds():
    """80 sentences at beam 16 over 33 tiles: 1280 rows x 32 tiles = 40960 (row, tile)
    pairs, more than the sort assembles in LDS (36864), so each pair is stored to its
    place directly; the result must still equal the plain scan."""
    shape = synth.ModelShape(64, 2, 256, 1, 1, 4200)
    blob = synth.make_weights(shape, seed=95, lively=True, eos_boost=1.5)
    ids, offs = synth.make_sentences(synth.DataSetup(80, "uniform", 2, 8, "uniform"), shape.vocab, seed=96)
    search = synth.SearchSetup(beam=16, len_penalty=0.6, max_len_a=1.0, max_len_b=3, token_budget=8192, prune=1)
    model = G.new_model(shape, blob, "f32")
    fused = _translate(model, ids, offs, search, True)
    plain = _translate(model, ids, offs, search, False)
    model.close()
    for a, b in zip(fused[0], plain[0]):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(fused[1], plain[1], rtol=1e-6, atol=1e-6)
