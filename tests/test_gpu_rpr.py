"""GPU parity of relative position representations in encoder self-attention (the
teachers' RPR, Sec. 3.1, maximum relative length 8) against the CPU oracle.

The tables are drawn large (std 0.5) so that the relative terms move the result well
beyond the tolerances.  Covers head sizes 32 and 64, fp32 and fp16, clip distances 1 and
8, a sentence longer than one 128-key softmax chunk, and the whole model
(teacher-forced logits).  Tolerances as in test_gpu_parity.
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

ENC_TOL = {"f32": 1e-4, "f16": 3e-2}
LOGIT_TOL = {"f32": 1e-3, "f16": 5e-2}


def _encoder_out(shape, blob, dtype, srcs):
    from paper_2109_08008_amd import nt
    model = G.new_model(shape, blob, dtype)
    st, _ = G.gpu_encode(model, srcs, synth.SearchSetup(beam=1, max_len_b=4))
    try:
        return nt.nt_dec_state_encoder_out(st, shape.d_model)
    finally:
        nt.nt_free_state(st)


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("d,H,rel_k", [(128, 4, 8), (256, 4, 8), (128, 4, 1)])
def test_encoder_output_with_relative_positions(d, H, rel_k, dtype):
    shape = synth.ModelShape(d, H, 4 * d, 2, 1, 203, rel_k=rel_k)
    blob = synth.make_weights(shape, seed=21, lively=True)
    rng = np.random.default_rng(6)
    srcs = [list(rng.integers(4, shape.vocab, size=n)) for n in (1, 5, 9, 17, 23, 40)]
    enc = _encoder_out(shape, blob, dtype, srcs)
    om = G.oracle_model(shape, blob, dtype)
    plain = G.oracle_model(synth.ModelShape(d, H, 4 * d, 2, 1, 203), _without_tables(shape, blob), dtype)
    err = moved = 0.0
    for b, s in enumerate(srcs):
        ref = om.encode(s)
        err = max(err, float(np.abs(enc[b, :len(s)] - ref).max()))
        moved = max(moved, float(np.abs(plain.encode(s) - ref).max()))
    print(f"d={d} k={rel_k} {dtype}: max abs err {err:.3g}; the tables move the output by {moved:.3g}")
    assert moved > 20 * max(err, ENC_TOL["f32"])   # the check can tell the tables apart
    assert err <= ENC_TOL[dtype]


def test_relative_positions_across_softmax_chunks():
    """S = 150: the query-key offsets span two 128-key chunks of the online softmax."""
    shape = synth.ModelShape(128, 4, 512, 1, 1, 203, rel_k=8)
    blob = synth.make_weights(shape, seed=22, lively=True)
    rng = np.random.default_rng(7)
    srcs = [list(rng.integers(4, shape.vocab, size=n)) for n in (150, 129, 3)]
    enc = _encoder_out(shape, blob, "f32", srcs)
    om = G.oracle_model(shape, blob, "f32")
    for b, s in enumerate(srcs):
        np.testing.assert_allclose(enc[b, :len(s)], om.encode(s), atol=ENC_TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_teacher_forced_logits_with_relative_positions(dtype):
    shape = synth.ModelShape(256, 4, 1024, 2, 1, 517, rel_k=8)
    blob = synth.make_weights(shape, seed=23, lively=True)
    rng = np.random.default_rng(8)
    srcs = [list(rng.integers(4, shape.vocab, size=n)) for n in (4, 12, 30)]
    tgts = [list(rng.integers(3, shape.vocab, size=int(rng.integers(1, 10)))) for _ in srcs]
    model = G.new_model(shape, blob, dtype)
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, dtype)
    err = max(float(np.abs(got[b] - om.teacher_forced_logits(s, tg)).max()) for b, (s, tg) in enumerate(zip(srcs, tgts)))
    print(f"{dtype}: teacher-forced logits max abs err {err:.3g}")
    assert err <= LOGIT_TOL[dtype]


def _without_tables(shape, blob):
    named = synth.unpack(shape, blob)
    plain = synth.ModelShape(shape.d_model, shape.n_heads, shape.d_ffn, shape.n_enc, shape.n_dec, shape.vocab)
    return synth.pack(plain, {n: x for n, x in named.items() if not n.endswith(("rel_k", "rel_v"))})
