"""ctypes binding of libnt.so, the C ABI declared in include/nt.h.

Argument marshalling only: every step of the translation path runs in the library's
HIP kernels.  torch supplies device memory (weight buffer, workspace) and the stream.
The functions keep the C names; :class:`Model` bundles a loaded model with its torch
weight buffer for convenience.  If libnt.so is missing or fails to load, every entry
point raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_void_p

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnt.so")

NT_OK, NT_E_INVALID, NT_E_UNSUPPORTED, NT_E_WORKSPACE, NT_E_DEVICE, NT_E_STATE, NT_E_NUMERIC = range(7)
NT_F32, NT_F16, NT_BF16 = 0, 1, 2
DTYPES = {"f32": NT_F32, "f16": NT_F16, "bf16": NT_BF16}
(NT_K_GEMM_ENC, NT_K_GEMM_DEC, NT_K_GEMM_VOCAB, NT_K_DLCL, NT_K_LN, NT_K_ATTN_ENC, NT_K_ATTN_SELF,
 NT_K_ATTN_CROSS, NT_K_SELECT, NT_K_SEARCH) = range(10)
KERNEL_CLASSES = ["gemm_enc", "gemm_dec", "gemm_vocab", "dlcl", "ln", "attn_enc", "attn_self", "attn_cross",
                  "select", "search"]

EXPORTS = [
    "nt_weights_size", "nt_load_weights", "nt_free_model", "nt_workspace_size", "nt_translate_workspace_size",
    "nt_encode", "nt_decode_step", "nt_dec_state_read", "nt_dec_state_info", "nt_dec_state_encoder_out",
    "nt_free_state", "nt_translate", "nt_last_error", "nt_prof_enable", "nt_prof_reset", "nt_prof_get",
    "nt_op_gemm", "nt_op_gemm_ln", "nt_prof_config", "nt_set_graphs", "nt_set_beam_fused", "nt_set_streams", "nt_prof_units", "nt_op_select",
    "nt_op_select_tiled", "nt_op_select_tiled_noalloc",
    "nt_ensemble", "nt_quantize_fp8",
]
NT_ENS_MEAN_LOGP, NT_ENS_LOG_MEAN_P = 0, 1
NT_SELECT_NOALLOC_MAX_RECORDS = 1 << 20   # include/nt.h: records of nt_op_select_tiled_noalloc


class nt_model_cfg(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("n_heads", c_int32), ("d_ffn", c_int32), ("n_enc", c_int32),
                ("n_dec", c_int32), ("vocab", c_int32), ("max_positions", c_int32), ("pad_id", c_int32),
                ("bos_id", c_int32), ("eos_id", c_int32), ("dtype", c_int32), ("dlcl_hist_norm", c_int32),
                ("ln_eps", c_float), ("rel_pos_k", c_int32), ("fp8_weights", c_int32), ("fp8_kv", c_int32)]


class nt_search_cfg(ctypes.Structure):
    _fields_ = [("beam", c_int32), ("len_penalty", c_float), ("max_len_a", c_float), ("max_len_b", c_int32),
                ("max_len_cap", c_int32), ("token_budget", c_int32), ("max_batch_sents", c_int32),
                ("early_stop", c_int32), ("prune", c_int32)]


class NTError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"nt status {status}: {message}")
        self.status = status
        self.message = message


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libnt.so (built by paper_2109_08008_amd.build) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2109_08008_amd.build.build_library()")
    # torch ships its own HIP runtime.  Loaded first, it provides the libamdhip64.so.7 that
    # libnt.so links against, so the process has one runtime and torch's device memory and
    # streams are valid here; loaded after libnt.so, it would bring a second runtime.
    import torch  # noqa: F401
    L = ctypes.CDLL(path)
    P = c_void_p
    sig = {
        "nt_weights_size": (c_int32, [POINTER(nt_model_cfg), POINTER(c_size_t), POINTER(c_size_t)]),
        "nt_load_weights": (c_int32, [POINTER(nt_model_cfg), POINTER(c_float), c_size_t, P, c_size_t, P, POINTER(P)]),
        "nt_free_model": (None, [P]),
        "nt_ensemble": (c_int32, [POINTER(P), c_int32, c_int32, POINTER(P)]),
        "nt_quantize_fp8": (c_int32, [POINTER(c_float), c_int32, c_int32, POINTER(ctypes.c_uint8), POINTER(c_float)]),
        "nt_workspace_size": (c_int32, [P, POINTER(nt_search_cfg), c_int32, c_int32, POINTER(c_size_t)]),
        "nt_translate_workspace_size": (c_int32, [P, POINTER(nt_search_cfg), POINTER(c_int64), c_int32,
                                                  POINTER(c_size_t)]),
        "nt_encode": (c_int32, [P, P, P, POINTER(c_int32), c_int32, c_int32, POINTER(nt_search_cfg), P, c_size_t, P,
                                POINTER(P)]),
        "nt_decode_step": (c_int32, [P, P, P, POINTER(c_int32), P]),
        "nt_dec_state_read": (c_int32, [P, POINTER(c_int32), POINTER(c_int32), POINTER(c_float), POINTER(c_float), P]),
        "nt_dec_state_info": (c_int32, [P] + [POINTER(c_int32)] * 6),
        "nt_dec_state_encoder_out": (c_int32, [P, POINTER(c_float), P]),
        "nt_free_state": (None, [P]),
        "nt_translate": (c_int32, [P, POINTER(nt_search_cfg), POINTER(c_int32), POINTER(c_int64), c_int32,
                                   POINTER(c_int32), c_int64, POINTER(c_int64), POINTER(c_float), POINTER(c_float),
                                   P, c_size_t, P]),
        "nt_last_error": (c_char_p, []),
        "nt_prof_enable": (c_int32, [c_uint32]),
        "nt_prof_config": (c_int32, [c_uint32, c_int32]),
        "nt_set_graphs": (c_int32, [c_int32]),
        "nt_set_beam_fused": (c_int32, [c_int32]),
        "nt_set_streams": (c_int32, [c_int32]),
        "nt_op_select": (c_int32, [P, c_int32, c_int32, c_int32, P, P, P, P]),
        "nt_op_select_tiled": (c_int32, [P, c_int32, c_int32, c_int32, P, P, P, P]),
        "nt_op_select_tiled_noalloc": (c_int32, [P, c_int32, c_int32, c_int32, P, P, P, P]),
        "nt_prof_units": (c_int32, [POINTER(c_int64), POINTER(c_int64)]),
        "nt_prof_reset": (c_int32, []),
        "nt_prof_get": (c_int32, [c_int32, POINTER(c_int64), POINTER(c_double), POINTER(c_double), POINTER(c_double)]),
        "nt_op_gemm": (c_int32, [c_int32, P, c_int32, P, c_int32, c_int32, c_int32, P, P, P, c_int32, c_int32, c_int32,
                                 c_int32, P, P]),
        "nt_op_gemm_ln": (c_int32, [c_int32, P, c_int32, P, c_int32, c_int32, c_int32, P, c_float, P, P, c_int32,
                                    c_int32, c_int32, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int):
    if status != NT_OK:
        raise NTError(status, load_library().nt_last_error().decode())


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(POINTER(ctype)) if a is not None else None


def _stream(stream):
    if stream is None:
        import torch
        return c_void_p(torch.cuda.current_stream().cuda_stream)
    return c_void_p(int(stream))


def model_cfg(shape, dtype: str = "f16", hist_norm: bool = True, ln_eps: float = 1e-5,
              pad_id: int = 0, bos_id: int = 1, eos_id: int = 2) -> nt_model_cfg:
    """nt_model_cfg from any object with d_model, n_heads, d_ffn, n_enc, n_dec, vocab, max_positions
    (and optionally rel_k).  dtype "f8" is the FP8 mode: fp16 activations, FP8 projection
    weights and an FP8 self-attention key/value cache; "f8w" is FP8 weights alone."""
    f8 = dtype in ("f8", "f8w")
    return nt_model_cfg(shape.d_model, shape.n_heads, shape.d_ffn, shape.n_enc, shape.n_dec, shape.vocab,
                        getattr(shape, "max_positions", 1024), pad_id, bos_id, eos_id, DTYPES["f16" if f8 else dtype],
                        1 if hist_norm else 0, ln_eps, int(getattr(shape, "rel_k", 0)), int(f8), int(dtype == "f8"))


def search_cfg(s) -> nt_search_cfg:
    """nt_search_cfg from any object with the nt_search_cfg field names."""
    return nt_search_cfg(int(s.beam), float(s.len_penalty), float(s.max_len_a), int(s.max_len_b),
                         int(getattr(s, "max_len_cap", 0)), int(s.token_budget), int(s.max_batch_sents),
                         int(s.early_stop), int(s.prune))


def max_target_tokens(sc: nt_search_cfg, src_len: int) -> int:
    """A sentence's target length limit under sc, as the library computes it."""
    n = int(np.floor(np.float32(sc.max_len_a) * np.float64(src_len))) + int(sc.max_len_b)
    return min(n, int(sc.max_len_cap)) if sc.max_len_cap > 0 else n


# ---- the C entry points ----------------------------------------------------------------
def nt_weights_size(cfg: nt_model_cfg):
    hf, db = c_size_t(), c_size_t()
    _check(load_library().nt_weights_size(ctypes.byref(cfg), ctypes.byref(hf), ctypes.byref(db)))
    return hf.value, db.value


def nt_load_weights(cfg: nt_model_cfg, host_weights: np.ndarray, device_buf: int, device_bytes: int, stream=None):
    w = np.ascontiguousarray(host_weights, dtype=np.float32)
    out = c_void_p()
    _check(load_library().nt_load_weights(ctypes.byref(cfg), _ptr(w, c_float), w.size, c_void_p(device_buf),
                                          device_bytes, _stream(stream), ctypes.byref(out)))
    return out


def nt_free_model(m):
    load_library().nt_free_model(m)


def nt_ensemble(members, rule: int):
    """Ensemble handle over member model handles (borrowed: they must outlive it)."""
    arr = (c_void_p * max(len(members), 1))(*[m.value if isinstance(m, c_void_p) else m for m in members])
    out = c_void_p()
    _check(load_library().nt_ensemble(arr, len(members), rule, ctypes.byref(out)))
    return out


def nt_workspace_size(m, search: nt_search_cfg, max_sents: int, max_src: int) -> int:
    b = c_size_t()
    _check(load_library().nt_workspace_size(m, ctypes.byref(search), max_sents, max_src, ctypes.byref(b)))
    return b.value


def nt_translate_workspace_size(m, search: nt_search_cfg, h_src_off: np.ndarray) -> int:
    off = np.ascontiguousarray(h_src_off, dtype=np.int64)
    b = c_size_t()
    _check(load_library().nt_translate_workspace_size(m, ctypes.byref(search), _ptr(off, c_int64), off.size - 1,
                                                      ctypes.byref(b)))
    return b.value


def nt_encode(m, d_src: int, d_len: int, h_len: np.ndarray, B: int, S: int, search: nt_search_cfg, d_ws: int,
              ws_bytes: int, stream=None):
    hl = None if h_len is None else np.ascontiguousarray(h_len, dtype=np.int32)
    st = c_void_p()
    _check(load_library().nt_encode(m, c_void_p(d_src), c_void_p(d_len), _ptr(hl, c_int32), B, S,
                                    ctypes.byref(search), c_void_p(d_ws), ws_bytes, _stream(stream),
                                    ctypes.byref(st)))
    return st


def nt_decode_step(st, d_forced: int | None = None, d_logits: int | None = None, stream=None) -> int:
    alive = c_int32()
    _check(load_library().nt_decode_step(st, c_void_p(d_forced) if d_forced else None,
                                         c_void_p(d_logits) if d_logits else None, ctypes.byref(alive),
                                         _stream(stream)))
    return alive.value


def nt_dec_state_info(st) -> dict:
    vals = [c_int32() for _ in range(6)]
    _check(load_library().nt_dec_state_info(st, *[ctypes.byref(v) for v in vals]))
    return dict(zip(["B", "S", "beam", "max_tgt", "steps", "alive"], [v.value for v in vals]))


def nt_dec_state_read(st, stream=None):
    info = nt_dec_state_info(st)
    B, T = info["B"], info["max_tgt"]
    toks = np.zeros((B, T), dtype=np.int32)
    lens = np.zeros(B, dtype=np.int32)
    scores = np.zeros(B, dtype=np.float32)
    logp = np.zeros((B, T), dtype=np.float32)
    _check(load_library().nt_dec_state_read(st, _ptr(toks, c_int32), _ptr(lens, c_int32), _ptr(scores, c_float),
                                            _ptr(logp, c_float), _stream(stream)))
    return ([toks[b, :lens[b]].copy() for b in range(B)], scores, [logp[b, :lens[b]].copy() for b in range(B)])


def nt_dec_state_encoder_out(st, d_model: int, stream=None) -> np.ndarray:
    info = nt_dec_state_info(st)
    out = np.zeros((info["B"], info["S"], d_model), dtype=np.float32)
    _check(load_library().nt_dec_state_encoder_out(st, _ptr(out, c_float), _stream(stream)))
    return out


def nt_free_state(st):
    load_library().nt_free_state(st)


def nt_translate(m, search: nt_search_cfg, h_src: np.ndarray, h_src_off: np.ndarray, out_cap: int, d_ws: int,
                 ws_bytes: int, stream=None):
    src = np.ascontiguousarray(h_src, dtype=np.int32)
    off = np.ascontiguousarray(h_src_off, dtype=np.int64)
    n = off.size - 1
    out = np.zeros(max(out_cap, 1), dtype=np.int32)
    out_off = np.zeros(n + 1, dtype=np.int64)
    score = np.zeros(n, dtype=np.float32)
    logp = np.zeros(max(out_cap, 1), dtype=np.float32)
    _check(load_library().nt_translate(m, ctypes.byref(search), _ptr(src, c_int32), _ptr(off, c_int64), n,
                                       _ptr(out, c_int32), out_cap, _ptr(out_off, c_int64), _ptr(score, c_float),
                                       _ptr(logp, c_float), c_void_p(d_ws), ws_bytes, _stream(stream)))
    return out[:out_off[-1]], out_off, score, logp[:out_off[-1]]


def nt_op_gemm(dtype: str, d_A: int, lda: int, d_Bt: int, M: int, N: int, K: int, d_bias, d_resid, d_out: int,
               ldc: int, out_f32: bool = False, relu: bool = False, tile: int = 0, d_bscale=None, stream=None):
    _check(load_library().nt_op_gemm(DTYPES[dtype], c_void_p(d_A), lda, c_void_p(d_Bt), M, N, K,
                                     c_void_p(d_bias) if d_bias else None, c_void_p(d_resid) if d_resid else None,
                                     c_void_p(d_out), ldc, int(out_f32), int(relu), tile,
                                     c_void_p(d_bscale) if d_bscale else None, _stream(stream)))


def nt_op_gemm_ln(dtype: str, d_A: int, lda: int, d_Bt: int, M: int, N: int, K: int, d_colsum: int, ln_eps: float,
                  d_bias, d_out: int, ldc: int, relu: bool = False, tile: int = 0, d_bscale=None, stream=None):
    _check(load_library().nt_op_gemm_ln(DTYPES[dtype], c_void_p(d_A), lda, c_void_p(d_Bt), M, N, K,
                                        c_void_p(d_colsum), float(ln_eps),
                                        c_void_p(d_bias) if d_bias else None, c_void_p(d_out), ldc, int(relu),
                                        tile, c_void_p(d_bscale) if d_bscale else None, _stream(stream)))


def nt_quantize_fp8(w: np.ndarray):
    """The library's FP8 weight quantization of an [in, out] fp32 matrix: (codes [out, in]
    uint8, scales [out] fp32)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    q = np.zeros((w.shape[1], w.shape[0]), dtype=np.uint8)
    sc = np.zeros(w.shape[1], dtype=np.float32)
    _check(load_library().nt_quantize_fp8(_ptr(w, c_float), w.shape[0], w.shape[1], _ptr(q, ctypes.c_uint8),
                                          _ptr(sc, c_float)))
    return q, sc


def nt_op_select(d_logits: int, rows: int, V: int, k: int, d_topv: int, d_topi: int, d_lse: int, stream=None):
    _check(load_library().nt_op_select(c_void_p(d_logits), rows, V, k, c_void_p(d_topv), c_void_p(d_topi),
                                       c_void_p(d_lse), _stream(stream)))


def nt_op_select_tiled(d_logits: int, rows: int, V: int, k: int, d_topv: int, d_topi: int, d_lse: int,
                       stream=None):
    _check(load_library().nt_op_select_tiled(c_void_p(d_logits), rows, V, k, c_void_p(d_topv), c_void_p(d_topi),
                                             c_void_p(d_lse), _stream(stream)))


def nt_op_select_tiled_noalloc(d_logits: int, rows: int, V: int, k: int, d_topv: int, d_topi: int, d_lse: int,
                               stream=None):
    _check(load_library().nt_op_select_tiled_noalloc(c_void_p(d_logits), rows, V, k, c_void_p(d_topv),
                                                     c_void_p(d_topi), c_void_p(d_lse), _stream(stream)))


def nt_prof_enable(mask: int):
    _check(load_library().nt_prof_enable(mask))


def nt_prof_config(mask: int, stride: int):
    _check(load_library().nt_prof_config(mask, stride))


def nt_set_graphs(enable: bool):
    _check(load_library().nt_set_graphs(int(bool(enable))))


def nt_set_beam_fused(enable: bool):
    _check(load_library().nt_set_beam_fused(int(bool(enable))))


def nt_set_streams(n: int):
    _check(load_library().nt_set_streams(int(n)))


def nt_prof_units() -> tuple:
    """(batch encodes, decoder steps) counted by nt_translate since nt_prof_config."""
    e, s = c_int64(), c_int64()
    _check(load_library().nt_prof_units(ctypes.byref(e), ctypes.byref(s)))
    return e.value, s.value


def nt_prof_reset():
    _check(load_library().nt_prof_reset())


def nt_prof_get(kernel_class: int) -> dict:
    n, ms, by, fl = c_int64(), c_double(), c_double(), c_double()
    _check(load_library().nt_prof_get(kernel_class, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(by),
                                      ctypes.byref(fl)))
    return {"launches": n.value, "ms": ms.value, "bytes": by.value, "flops": fl.value}


# ---- convenience wrappers ---------------------------------------------------------------
class _Translator:
    """nt_translate over a handle, with a cached torch workspace (the per-call memory pool)."""

    handle = None
    device = None
    _ws = None

    def workspace(self, nbytes: int):
        """A cached torch byte buffer of at least nbytes."""
        import torch
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = None
            self._ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self._ws

    def translate(self, ids: np.ndarray, offs: np.ndarray, search):
        """Translate CSR sentences; returns (list of token arrays, scores, list of per-token log-probs)."""
        sc = search_cfg(search)
        need = nt_translate_workspace_size(self.handle, sc, offs)
        ws = self.workspace(need)
        lens = np.diff(offs)
        cap = int(sum(max_target_tokens(sc, int(L)) for L in lens))
        out, out_off, score, logp = nt_translate(self.handle, sc, ids, offs, cap, ws.data_ptr(), ws.numel())
        n = len(lens)
        return ([out[out_off[i]:out_off[i + 1]] for i in range(n)], score,
                [logp[out_off[i]:out_off[i + 1]] for i in range(n)])

    def close(self):
        if getattr(self, "handle", None):
            nt_free_model(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Model(_Translator):
    """A model loaded on the current CUDA (HIP) device; owns its torch weight buffer."""

    def __init__(self, shape, blob: np.ndarray, dtype: str = "f16", hist_norm: bool = True, device=None):
        import torch
        self.shape = shape
        self.dtype = dtype
        self.cfg = model_cfg(shape, dtype, hist_norm)
        self.host_floats, self.device_bytes = nt_weights_size(self.cfg)
        if blob.size != self.host_floats:
            raise ValueError(f"blob has {blob.size} floats, model needs {self.host_floats}")
        self.device = torch.device(device or "cuda")
        self.buf = torch.empty(self.device_bytes, dtype=torch.uint8, device=self.device)
        self.handle = nt_load_weights(self.cfg, blob, self.buf.data_ptr(), self.device_bytes)
        self._ws = None


class Ensemble(_Translator):
    """Ensemble decoding over loaded Models (kept alive here for the handle's lifetime)."""

    def __init__(self, members: list, rule: int = NT_ENS_MEAN_LOGP):
        self.members = list(members)
        self.rule = rule
        self.device = self.members[0].device
        self.handle = nt_ensemble([m.handle for m in self.members], rule)
        self._ws = None
