"""Band attention (streaming attention and low-latency streaming attention) for
AMD Instinct MI355X (gfx950).

The compute lives in a C-ABI shared library (``libsa.so``, declared in
``include/sa.h``) built from the HIP sources under ``csrc/``; this package only
marshals torch tensors into that ABI (see :mod:`.binding`, imported on first
use of one of its names).
"""

_BINDING_NAMES = {
    "SA_BF16", "SA_F32", "SAError", "library_path", "load_library", "sa_forward",
    "sa_backward", "llsa_forward", "llsa_backward", "llsa_paper_forward",
    "llsa_paper_backward", "sa_stream_step", "StreamState", "llsa_stream_step",
    "LlsaStreamState",
}


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import binding

        return getattr(binding, name)
    raise AttributeError(name)
