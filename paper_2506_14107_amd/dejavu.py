"""Python binding of libdejavu.so (argument marshalling only).

The functions named like the C entry points (``dv_create``, ``dv_encode``, ...) take
plain integers for device pointers and streams and raise ``DejaVuError`` on a
non-zero status.  ``Encoder`` wraps them for torch tensors: torch supplies device
memory and the current HIP stream; every step of the computation runs in the
library's HIP kernels.  Importing this module never falls back to anything: if
the library is missing, ``load()`` raises.
"""
import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libdejavu.so")

DV_OK, DV_EINVAL, DV_ENOMEM, DV_EHIP, DV_EUNSUPPORTED = 0, -1, -2, -3, -4
DV_F32, DV_BF16 = 0, 1
STAGES = ["patch", "gate", "compact", "ln1", "qkv", "attn", "oproj", "ln2", "fc1", "fc2",
          "merge", "final", "restore", "cls"]
DV_FLAG_RESTORE = 1
DV_FLAG_DECISION = 2
DV_FLAG_REORDER = 4


class DejaVuError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"dejavu error {code}: {msg}")
        self.code = code


class dv_config(ctypes.Structure):
    _fields_ = [("image_size", ctypes.c_int), ("patch", ctypes.c_int), ("depth", ctypes.c_int),
                ("width", ctypes.c_int), ("heads", ctypes.c_int), ("mlp", ctypes.c_int),
                ("dtype", ctypes.c_int), ("max_batch_frames", ctypes.c_int),
                ("flags", ctypes.c_uint)]


_lib = None
_P = ctypes.c_void_p


def load(path=None):
    """Load libdejavu.so (built by ``paper_2506_14107_amd.build``); raises if it is absent."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise FileNotFoundError(f"{p} is missing: build it with python -m paper_2506_14107_amd.build")
    lib = ctypes.CDLL(p)
    sig = {
        "dv_weights_floats": (ctypes.c_size_t, [ctypes.POINTER(dv_config)]),
        "dv_create": (ctypes.c_int, [ctypes.POINTER(dv_config), _P, ctypes.c_size_t,
                                     ctypes.POINTER(_P)]),
        "dv_destroy": (ctypes.c_int, [_P]),
        "dv_last_error": (ctypes.c_char_p, []),
        "dv_workspace_bytes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
        "dv_encode": (ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_float, _P, _P,
                                     _P]),
        "dv_encode_noalloc": (ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                             _P, _P, _P]),
        "dv_encode_masked": (ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, _P, _P, _P, _P]),
        "dv_encode_tokens": (ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                            _P, _P, _P, _P, _P]),
        "dv_compact": (ctypes.c_int, [_P, ctypes.c_int, ctypes.c_int, ctypes.c_int, _P, _P, _P,
                                      _P, _P]),
        "dv_stream_encode": (ctypes.c_int, [_P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                            _P, _P, _P, _P, _P]),
        "dv_stream_reset": (ctypes.c_int, [_P]),
        "dv_stream_held": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int)]),
        "dv_stream_flush": (ctypes.c_int, [_P, _P, _P, _P, _P]),
        "dv_mfma_probe": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, _P,
                                         ctypes.POINTER(ctypes.c_double), _P]),
        "dv_profile": (ctypes.c_int, [_P, ctypes.c_uint]),
        "dv_profile_read": (ctypes.c_int, [_P, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_longlong)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    if path is None:
        _lib = lib
    return lib


def _check(rc):
    if rc != DV_OK:
        raise DejaVuError(rc, load().dv_last_error().decode())


def make_config(image_size, patch, depth, width, heads, mlp, dtype, max_batch_frames, flags=0):
    dt = {"f32": DV_F32, "bf16": DV_BF16}.get(dtype, dtype)
    return dv_config(image_size, patch, depth, width, heads, mlp, dt, max_batch_frames, flags)


# ---- the C entry points, one to one -----------------------------------------------------------
def dv_weights_floats(cfg):
    return load().dv_weights_floats(ctypes.byref(cfg))


def dv_create(cfg, weights):
    """weights: host float32 array (the blob).  Returns the handle (an int)."""
    w = np.ascontiguousarray(weights, dtype=np.float32)
    h = _P()
    _check(load().dv_create(ctypes.byref(cfg), w.ctypes.data, w.nbytes, ctypes.byref(h)))
    return h.value


def dv_destroy(handle):
    _check(load().dv_destroy(handle))


def dv_last_error():
    return load().dv_last_error().decode()


def dv_workspace_bytes(handle):
    n = ctypes.c_size_t()
    _check(load().dv_workspace_bytes(handle, ctypes.byref(n)))
    return n.value


def dv_encode(handle, frames, n_frames, group_size, tau, out_embeddings, out_masks, stream):
    _check(load().dv_encode(handle, frames, n_frames, group_size, tau, out_embeddings,
                            out_masks, stream))


def dv_encode_noalloc(handle, frames, n_frames, group_size, tau, out_embeddings, out_masks,
                      stream):
    _check(load().dv_encode_noalloc(handle, frames, n_frames, group_size, tau, out_embeddings,
                                    out_masks, stream))


DV_SCRATCH_BYTES = 128 << 20   # the static scratch array of dv_encode_noalloc


def dv_encode_masked(handle, frames, n_frames, group_size, masks, out_embeddings, out_masks,
                     stream):
    _check(load().dv_encode_masked(handle, frames, n_frames, group_size, masks, out_embeddings,
                                   out_masks, stream))


def dv_encode_tokens(handle, frames, n_frames, group_size, tau, masks, out_embeddings, out_masks,
                     out_tokens, stream):
    _check(load().dv_encode_tokens(handle, frames, n_frames, group_size, tau, masks,
                                   out_embeddings, out_masks, out_tokens, stream))


def dv_stream_encode(handle, frames, n_frames, group_size, tau, masks, out_embeddings, out_masks,
                     out_tokens, stream):
    _check(load().dv_stream_encode(handle, frames, n_frames, group_size, tau, masks,
                                   out_embeddings, out_masks, out_tokens, stream))


def dv_stream_reset(handle):
    _check(load().dv_stream_reset(handle))


def dv_stream_held(handle):
    n = ctypes.c_int(0)
    _check(load().dv_stream_held(handle, ctypes.byref(n)))
    return n.value


def dv_stream_flush(handle, out_embeddings, out_masks, out_tokens, stream):
    _check(load().dv_stream_flush(handle, out_embeddings, out_masks, out_tokens, stream))


def dv_compact(masks, n_frames, n_tokens, group_size, idx, pos, qoff, count, stream):
    _check(load().dv_compact(masks, n_frames, n_tokens, group_size, idx, pos, qoff, count,
                             stream))


def dv_mfma_probe(blocks, iters, sink, stream):
    """Enqueues the MFMA-loop probe; returns the FLOPs of the launch."""
    fl = ctypes.c_double()
    _check(load().dv_mfma_probe(blocks, iters, sink, ctypes.byref(fl), stream))
    return fl.value


DV_PROFILE_ALL = 0x3FFF


def dv_profile(handle, stage_mask):
    _check(load().dv_profile(handle, int(stage_mask)))


def dv_profile_read(handle, stage):
    ms, n = ctypes.c_double(), ctypes.c_longlong()
    _check(load().dv_profile_read(handle, stage, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ---- torch convenience wrapper ----------------------------------------------------------------
def _ptr(t):
    return 0 if t is None else t.data_ptr()


def _stream(stream):
    import torch
    return (stream or torch.cuda.current_stream()).cuda_stream


class Encoder:
    """A handle bound to one model.  Tensors must live on the current HIP device."""

    def __init__(self, model, weights, max_batch_frames):
        m = model
        self.model = m
        flags = (DV_FLAG_RESTORE if getattr(m, "restore", False) else 0) | \
            (DV_FLAG_DECISION if getattr(m, "decision", False) else 0) | \
            (DV_FLAG_REORDER if getattr(m, "reorder", False) else 0)
        self.cfg = make_config(m.image_size, m.patch, m.depth, m.width, m.heads, m.mlp, m.dtype,
                               max_batch_frames, flags)
        self.handle = dv_create(self.cfg, weights)

    def close(self):
        if self.handle:
            dv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _outs(self, n, want_masks, want_tokens):
        import torch
        m = self.model
        emb = torch.empty((n, m.width), dtype=torch.float32, device="cuda")
        masks = (torch.empty((n, m.depth, m.n_tokens), dtype=torch.uint8, device="cuda")
                 if want_masks else None)
        toks = (torch.empty((n, m.n_tokens, m.width), dtype=torch.float32, device="cuda")
                if want_tokens else None)
        return emb, masks, toks

    def _check_frames(self, frames):
        m = self.model
        if (not frames.is_cuda or frames.dtype.itemsize != 4 or not frames.is_contiguous()
                or tuple(frames.shape[1:]) != (3, m.image_size, m.image_size)):
            raise ValueError("frames must be a contiguous fp32 CUDA tensor [n, 3, S, S]")

    def encode(self, frames, group_size, tau, want_masks=True, want_tokens=False, stream=None):
        """Gate mode; returns (embeddings, masks or None, tokens or None)."""
        self._check_frames(frames)
        n = frames.shape[0]
        emb, masks, toks = self._outs(n, want_masks, want_tokens)
        if want_tokens:
            dv_encode_tokens(self.handle, _ptr(frames), n, group_size, float(tau), 0, _ptr(emb),
                             _ptr(masks), _ptr(toks), _stream(stream))
        else:
            dv_encode(self.handle, _ptr(frames), n, group_size, float(tau), _ptr(emb),
                      _ptr(masks), _stream(stream))
        return emb, masks, toks

    def encode_noalloc(self, frames, group_size, tau, out_embeddings, out_masks=None, stream=None):
        """Gate mode through dv_encode_noalloc, into caller-allocated outputs (embeddings
        [n, D] fp32, masks [n, depth, N] uint8 or None); the library allocates nothing."""
        self._check_frames(frames)
        n = frames.shape[0]
        dv_encode_noalloc(self.handle, _ptr(frames), n, group_size, float(tau),
                          _ptr(out_embeddings), _ptr(out_masks), _stream(stream))
        return out_embeddings, out_masks

    def encode_masked(self, frames, group_size, masks_in, want_masks=True, want_tokens=False,
                      stream=None):
        """Mask-injection mode; masks_in: uint8 CUDA tensor [n, depth, N]."""
        self._check_frames(frames)
        n = frames.shape[0]
        m = self.model
        if (not masks_in.is_cuda or masks_in.dtype.itemsize != 1 or not masks_in.is_contiguous()
                or tuple(masks_in.shape) != (n, m.depth, m.n_tokens)):
            raise ValueError("masks must be a contiguous uint8 CUDA tensor [n, depth, N]")
        emb, masks, toks = self._outs(n, want_masks, want_tokens)
        if want_tokens:
            dv_encode_tokens(self.handle, _ptr(frames), n, group_size, 0.0, _ptr(masks_in),
                             _ptr(emb), _ptr(masks), _ptr(toks), _stream(stream))
        else:
            dv_encode_masked(self.handle, _ptr(frames), n, group_size, _ptr(masks_in), _ptr(emb),
                             _ptr(masks), _stream(stream))
        return emb, masks, toks

    def stream_encode(self, frames, group_size, tau=0.0, masks_in=None, want_masks=True,
                      want_tokens=False, stream=None):
        """The next frames of a stream (gate mode with tau, or injected masks_in).  Returns the
        outputs of the frames the call completes: its own frames, except that a reordered
        stream first completes the frames it held and then holds back those after its last
        anchor."""
        self._check_frames(frames)
        n = frames.shape[0]
        held = dv_stream_held(self.handle)
        emb, masks, toks = self._outs(n + held, want_masks, want_tokens)
        dv_stream_encode(self.handle, _ptr(frames), n, group_size, float(tau),
                         _ptr(masks_in) if masks_in is not None else 0, _ptr(emb), _ptr(masks),
                         _ptr(toks), _stream(stream))
        k = n + held - dv_stream_held(self.handle)
        return tuple(o[:k] if o is not None else None for o in (emb, masks, toks))

    def stream_flush(self, want_masks=True, want_tokens=False, stream=None):
        """End the stream: the outputs of the frames it still held (none without reordering)."""
        held = dv_stream_held(self.handle)
        emb, masks, toks = self._outs(held, want_masks, want_tokens)
        dv_stream_flush(self.handle, _ptr(emb) if held else 0, _ptr(masks) if held else 0,
                        _ptr(toks) if held else 0, _stream(stream))
        return emb, masks, toks

    def stream_reset(self):
        dv_stream_reset(self.handle)

    def profile(self, stages=True):
        """stages: True (all), False (off), or an iterable of stage names."""
        if stages is True:
            mask = DV_PROFILE_ALL
        elif not stages:
            mask = 0
        else:
            mask = sum(1 << STAGES.index(s) for s in stages)
        dv_profile(self.handle, mask)

    def profile_read(self):
        return {name: dv_profile_read(self.handle, i) for i, name in enumerate(STAGES)}


def compact(masks, group_size, stream=None):
    """Stream compaction of a [n_frames, n_tokens] uint8 CUDA map; returns (idx, pos, qoff, count)."""
    import torch
    F, N = masks.shape
    idx = torch.empty(F * N, dtype=torch.int32, device="cuda")
    pos = torch.empty(F * N, dtype=torch.int32, device="cuda")
    qoff = torch.empty(F + 1, dtype=torch.int32, device="cuda")
    cnt = torch.empty(1, dtype=torch.int32, device="cuda")
    dv_compact(_ptr(masks.contiguous()), F, N, group_size, _ptr(idx), _ptr(pos), _ptr(qoff),
               _ptr(cnt), _stream(stream))
    return idx, pos, qoff, cnt
