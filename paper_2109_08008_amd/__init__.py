"""MI355X (gfx950) implementation of the NiuTrans deep-encoder / shallow-decoder translation
path: DLCL encoder, cached incremental decoder, greedy/beam search, batch pruning and
dynamic batching, as hand-written HIP kernels behind the C ABI in include/nt.h.

``paper_2109_08008_amd.nt`` is the ctypes binding of that library (libnt.so, built by
``paper_2109_08008_amd.build``)."""
from . import nt  # noqa: F401
