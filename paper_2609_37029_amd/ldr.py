"""Python binding of libldr.so (include/ldr.h): argument marshalling only.

Every computation of the drafting step runs in the library's HIP kernels;
this module turns torch tensors (device memory, streams) into the C ABI's
pointers and sizes. It raises if the library is missing: there is no other
implementation behind these names.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libldr.so")

LDR_OK, LDR_EINVAL, LDR_ERANGE, LDR_EHIP, LDR_ENOMEM, LDR_ESCRATCH = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 16 << 20   # LDR_NOALLOC_SCRATCH_BYTES
LDR_F32, LDR_BF16 = 0, 1


class LdrError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {_lib().ldr_strerror(code).decode()} ({code})")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_q_heads", "n_kv_heads", "head_dim", "mlp", "vocab", "n_layers",
        "n_feat_layers", "block", "window", "summary", "dtype")] + [
        ("rope_theta", ctypes.c_float), ("ntk_alpha", ctypes.c_float),
        ("rms_eps", ctypes.c_float), ("drop_views", ctypes.c_int32),
        ("pool_slots", ctypes.c_int32), ("pool_stride", ctypes.c_int32 * 2)]

# ldr_view_drop bits (ablation variants)
LDR_DROP_WINDOW, LDR_DROP_SUMMARY, LDR_DROP_BOUNDARY = 1, 2, 4


LAYER_KEYS = ("in_norm", "wqkv", "q_norm", "k_norm", "wo", "post_norm", "w_gate_up", "w_down")
TOP_KEYS = ("embed", "mask_emb", "pos_emb", "fc_w", "fc_norm", "final_norm", "lm_head")


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_KEYS]


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in TOP_KEYS] + [
        ("layers", ctypes.POINTER(LayerWeights)), ("lm_head_tiled", ctypes.c_void_p)]


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_37029_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ, U64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t,
                                ctypes.c_uint64)
        CP = ctypes.POINTER(Config)
        sig = {
            "ldr_views_state_bytes": (SZ, [CP]),
            "ldr_views_stride_bytes": (SZ, [CP]),
            "ldr_views_layout": (ctypes.c_int, [CP, ctypes.POINTER(SZ)]),
            "ldr_workspace_bytes": (SZ, [CP, I32]),
            "ldr_tiled_bytes": (SZ, [I32, I32]),
            "ldr_tile_matrix": (ctypes.c_int, [P, I32, I32, I64, P, SZ, P]),
            "ldr_config_check": (ctypes.c_int, [CP]),
            "ldr_views_init": (ctypes.c_int, [ctypes.POINTER(P), CP, I32, P, P, P, P, I32, P, P,
                                              P, P]),
            "ldr_views_update": (ctypes.c_int, [P, P, I32, P, P, P, P]),
            "ldr_views_status": (ctypes.c_int, [P, ctypes.c_int, P]),
            "ldr_views_destroy": (None, [P]),
            "ldr_draft_step": (ctypes.c_int, [P, ctypes.POINTER(Weights), P, P, P, SZ, P]),
            "ldr_draft_step_launches": (I32, [CP, P, I32]),
            "ldr_draft_step_events": (ctypes.c_int, [P, ctypes.POINTER(Weights), P, P, P, SZ, P,
                                                     I32, P]),
            "ldr_sample_workspace_bytes": (SZ, [I32, I32]),
            "ldr_sample": (ctypes.c_int, [P, I32, I32, ctypes.c_float, I32, U64, U64, P, P, P, P,
                                          SZ, P]),
            "ldr_gumbel_fill": (ctypes.c_int, [U64, U64, I32, I32, I32, P, P]),
            "ldr_sample_noalloc": (ctypes.c_int, [P, I32, I32, ctypes.c_float, I32, U64, U64, P, P,
                                                  P, P]),
            "ldr_sample_markov": (ctypes.c_int, [P, I32, I32, I32, P, P, P, I32, I32,
                                                 ctypes.c_float, I32, U64, U64, P, P, P, P, SZ,
                                                 P]),
            "ldr_draft_step_sample_workspace_bytes": (SZ, [P, I32]),
            "ldr_draft_step_sample": (ctypes.c_int, [P, P, P, P, ctypes.c_float, U64, U64, P, P,
                                                     P, P, SZ, P]),
            "ldr_verify_workspace_bytes": (SZ, [I32, I32, I32]),
            "ldr_verify": (ctypes.c_int, [P, P, P, P, I32, I32, I32, ctypes.c_float, I32, U64,
                                          U64, P, P, P, P, SZ, P]),
            "ldr_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _LIB = L
    return _LIB


def lib():
    """The loaded ctypes library (raises if it was not built)."""
    return _lib()


def _check(rc: int, what: str):
    if rc != LDR_OK:
        raise LdrError(rc, what)


def config(shape) -> Config:
    """ldr_config of a synth.Shape-like object."""
    strides = tuple(getattr(shape, "pool_strides", ()) or (0, 0))
    return Config(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.mlp,
                  shape.vocab, shape.n_layers, shape.n_feat_layers, shape.block, shape.window,
                  shape.summary, LDR_BF16 if shape.dtype == "bf16" else LDR_F32,
                  shape.rope_theta, shape.ntk_alpha, shape.rms_eps,
                  getattr(shape, "drop_views", 0), getattr(shape, "pool_slots", 0) or 0,
                  (ctypes.c_int32 * 2)(*strides))


def state_bytes(shape) -> int:
    return _lib().ldr_views_state_bytes(ctypes.byref(config(shape)))


def stride_bytes(shape) -> int:
    return _lib().ldr_views_stride_bytes(ctypes.byref(config(shape)))


def layout(shape):
    off = (ctypes.c_size_t * 5)()
    _check(_lib().ldr_views_layout(ctypes.byref(config(shape)), off), "ldr_views_layout")
    return dict(zip(("kw", "vw", "m", "eta", "h"), list(off)))


def workspace_bytes(shape, batch: int) -> int:
    return _lib().ldr_workspace_bytes(ctypes.byref(config(shape)), batch)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Views:
    """The fixed-size views of `batch` sequences in one device arena."""

    def __init__(self, shape, batch: int, G: torch.Tensor, device="cuda", stream=None):
        self.shape, self.batch = shape, batch
        self.cfg = config(shape)
        self.stride = stride_bytes(shape)
        self.layout = layout(shape)
        self.arena = torch.empty(batch * self.stride, dtype=torch.uint8, device=device)
        self.pos = torch.empty(batch, dtype=torch.int64, device=device)
        self.G = G
        self._h = ctypes.c_void_p()
        self._stream = stream

    def init(self, n_prefix=None, K=None, V=None, h=None):
        """ldr_views_init: reset, then (if given) ingest a first prefix chunk."""
        maxp = 0 if K is None else K.shape[1]
        _check(_lib().ldr_views_init(ctypes.byref(self._h), ctypes.byref(self.cfg), self.batch,
                                     _ptr(self.arena), _ptr(self.pos), _ptr(self.G),
                                     _ptr(n_prefix), maxp, _ptr(K), _ptr(V), _ptr(h),
                                     _stream(self._stream)), "ldr_views_init")
        return self

    def update(self, n_new: torch.Tensor, K: torch.Tensor, V: torch.Tensor, h: torch.Tensor):
        """ldr_views_update with K/V [batch][max_new][D][Hkv][d], h [batch][L_b][hidden]."""
        _check(_lib().ldr_views_update(self._h, _ptr(n_new), K.shape[1], _ptr(K), _ptr(V),
                                       _ptr(h), _stream(self._stream)), "ldr_views_update")

    def status(self, clear: bool = False) -> int:
        return _lib().ldr_views_status(self._h, int(clear), _stream(self._stream))

    @property
    def handle(self):
        return self._h

    # Tensor views into the arena (for checks and snapshots).
    def _region(self, off, shape, dtype):
        el = torch.tensor([], dtype=dtype).element_size()
        n = 1
        for s in shape:
            n *= s
        per = self.arena.view(self.batch, self.stride)
        return per[:, off:off + n * el].view(dtype).view(self.batch, *shape)

    def _drops(self, bit) -> bool:
        return bool(getattr(self.shape, "drop_views", 0) & bit)

    def _pool(self) -> int:
        return 0 if self._drops(LDR_DROP_SUMMARY) else int(getattr(self.shape, "pool_slots", 0)
                                                           or 0)

    def _rows(self):
        """(window rows kept, rows per (layer, group) region) and the region as
        K [batch][D][Hkv][rows][d] and V [batch][D][Hkv][rows][d] (a transposed
        view of the stored V^T)."""
        s = self.shape
        wr = 0 if self._drops(LDR_DROP_WINDOW) else s.window
        wx = wr + 2 * self._pool()
        shp = (s.n_layers, s.n_kv_heads, wx, s.head_dim)
        vt = (s.n_layers, s.n_kv_heads, s.head_dim, wx)
        return wr, (self._region(self.layout["kw"], shp, s.torch_dtype),
                    self._region(self.layout["vw"], vt, s.torch_dtype).transpose(-1, -2))

    def window(self):
        """Window K and V as [batch][D][Hkv][W][d] (V is stored transposed,
        [D][Hkv][d][W]; this returns a transposed view of it); None without
        the window view."""
        if self._drops(LDR_DROP_WINDOW):
            return None
        wr, (K, V) = self._rows()
        return K[..., :wr, :], V[..., :wr, :]

    def pooled(self):
        """Slot means of the mean-pooled summary's two banks, K and V each
        [batch][2][D][Hkv][P][d]; None with the learned summary."""
        P = self._pool()
        if not P:
            return None
        wr, (K, V) = self._rows()
        return (torch.stack([K[..., wr + i * P:wr + (i + 1) * P, :] for i in range(2)], 1),
                torch.stack([V[..., wr + i * P:wr + (i + 1) * P, :] for i in range(2)], 1))

    def summary(self):
        if self._drops(LDR_DROP_SUMMARY) or self._pool():
            return None
        s = self.shape
        return (self._region(self.layout["m"], (s.n_layers, s.n_q_heads, s.summary, s.head_dim),
                             torch.float32),
                self._region(self.layout["eta"], (s.n_layers, s.n_q_heads, s.summary),
                             torch.float32))

    def boundary(self):
        if self._drops(LDR_DROP_BOUNDARY):
            return None
        s = self.shape
        return self._region(self.layout["h"], (s.n_feat_layers, s.hidden), s.torch_dtype)

    def close(self):
        if self._h:
            _lib().ldr_views_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tiled_bytes(rows: int, cols: int) -> int:
    return _lib().ldr_tiled_bytes(rows, cols)


def tile_matrix(m: torch.Tensor, stream=None) -> torch.Tensor:
    """ldr_tile_matrix of a row-major bf16 [rows][cols] device tensor: a flat
    bf16 tensor in the library's 256 x 32 tiled layout."""
    rows, cols = m.shape
    out = torch.empty(tiled_bytes(rows, cols) // 2, dtype=torch.bfloat16, device=m.device)
    _check(_lib().ldr_tile_matrix(_ptr(m), rows, cols, m.stride(0), _ptr(out),
                                  out.numel() * 2, _stream(stream)), "ldr_tile_matrix")
    return out


class DraftWeights:
    """ldr_weights over a synth weight dict of device tensors (kept alive here).
    tiled_head: also give the library a tiled copy of the vocabulary head."""

    def __init__(self, w: Dict, tiled_head: bool = False):
        self.w = w
        n = len(w["layers"])
        self._layers = (LayerWeights * n)()
        for j, L in enumerate(w["layers"]):
            for k in LAYER_KEYS:
                setattr(self._layers[j], k, L[k].data_ptr())
        self.head_tiled = tile_matrix(w["lm_head"]) if tiled_head else None
        self.c = Weights(*[w[k].data_ptr() for k in TOP_KEYS],
                         ctypes.cast(self._layers, ctypes.POINTER(LayerWeights)),
                         None if self.head_tiled is None else self.head_tiled.data_ptr())


def draft_step(views: Views, weights: DraftWeights, anchor: torch.Tensor,
               logits: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
               stream=None) -> torch.Tensor:
    """ldr_draft_step: base logits fp32 [batch][B][V]."""
    s = views.shape
    if logits is None:
        logits = torch.empty(views.batch, s.block, s.vocab, dtype=torch.float32,
                             device=views.arena.device)
    if workspace is None:
        workspace = torch.empty(workspace_bytes(s, views.batch), dtype=torch.uint8,
                                device=views.arena.device)
    _check(_lib().ldr_draft_step(views.handle, ctypes.byref(weights.c), _ptr(anchor),
                                 _ptr(logits), _ptr(workspace), workspace.numel(),
                                 _stream(stream)), "ldr_draft_step")
    return logits


LAUNCH_KINDS = ("fc_gemm", "slot_init", "qkv_gemm", "attention", "o_gemm", "post_norm",
                "gate_up_gemm", "down_gemm", "next_norm", "lm_head", "qkv_finish")


def draft_launches(shape):
    """Kinds (names) of the kernel launches of one draft step, in order."""
    cfg = config(shape)
    n = _lib().ldr_draft_step_launches(ctypes.byref(cfg), None, 0)
    kinds = (ctypes.c_int32 * n)()
    _lib().ldr_draft_step_launches(ctypes.byref(cfg), kinds, n)
    return [LAUNCH_KINDS[k] for k in kinds]


def draft_step_events(views: Views, weights: DraftWeights, anchor: torch.Tensor,
                      logits: torch.Tensor, workspace: torch.Tensor, events, stream=None):
    """ldr_draft_step recording raw hipEvent_t handles (ints or None) around its
    launches: events[i] before launch i, events[n] after the last."""
    arr = (ctypes.c_void_p * len(events))(*[e if e else None for e in events])
    _check(_lib().ldr_draft_step_events(views.handle, ctypes.byref(weights.c), _ptr(anchor),
                                        _ptr(logits), _ptr(workspace), workspace.numel(),
                                        arr, len(events), _stream(stream)),
           "ldr_draft_step_events")


class HipEvents:
    """hipEvent_t handles from the HIP runtime this process already loaded
    (the one torch uses), for timing single kernels on a stream. They are
    created without the system-scope fence an event record performs by
    default (an L2 write-back and invalidate that costs the following kernels
    several µs): timing only, read after the device has synchronised."""

    DISABLE_SYSTEM_FENCE = 0x20000000   # hipEventDisableSystemFence

    def __init__(self):
        path = None
        for line in open("/proc/self/maps"):
            if "libamdhip64" in line:
                path = line.split()[-1]
                break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded (initialise torch.cuda first)")
        self.rt = ctypes.CDLL(path)
        self.rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
        self.rt.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._made = []

    def create(self):
        e = ctypes.c_void_p()
        if self.rt.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        self._made.append(e.value)
        return e.value

    def record(self, e, stream=None):
        if self.rt.hipEventRecord(e, _stream(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, a, b) -> float:
        self.rt.hipEventSynchronize(b)
        ms = ctypes.c_float()
        if self.rt.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for e in self._made:
            self.rt.hipEventDestroy(e)
        self._made = []


def sample_workspace_bytes(rows: int, vocab: int) -> int:
    return _lib().ldr_sample_workspace_bytes(rows, vocab)


def sample(logits: torch.Tensor, temperature: float, top_k: int, seed: int, step: int,
           out=None, workspace: Optional[torch.Tensor] = None, stream=None):
    """ldr_sample over a [rows][V] fp32 tensor: (tokens int32, lse fp32, logq fp32)."""
    V = logits.shape[-1]
    rows = logits.numel() // V
    dev = logits.device
    if out is None:
        out = (torch.empty(rows, dtype=torch.int32, device=dev),
               torch.empty(rows, dtype=torch.float32, device=dev),
               torch.empty(rows, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = torch.empty(sample_workspace_bytes(rows, V), dtype=torch.uint8, device=dev)
    tok, lse, logq = out
    _check(_lib().ldr_sample(_ptr(logits), rows, V, float(temperature), int(top_k), int(seed),
                             int(step), _ptr(tok), _ptr(lse), _ptr(logq), _ptr(workspace),
                             workspace.numel(), _stream(stream)), "ldr_sample")
    return out


def sample_noalloc(logits: torch.Tensor, temperature: float, top_k: int, seed: int, step: int,
                   out=None, stream=None):
    """ldr_sample_noalloc: ldr_sample with the library's static device scratch
    in place of a workspace (no device allocation by the library)."""
    V = logits.shape[-1]
    rows = logits.numel() // V
    dev = logits.device
    if out is None:
        out = (torch.empty(rows, dtype=torch.int32, device=dev),
               torch.empty(rows, dtype=torch.float32, device=dev),
               torch.empty(rows, dtype=torch.float32, device=dev))
    tok, lse, logq = out
    _check(_lib().ldr_sample_noalloc(_ptr(logits), rows, V, float(temperature), int(top_k),
                                     int(seed), int(step), _ptr(tok), _ptr(lse), _ptr(logq),
                                     _stream(stream)), "ldr_sample_noalloc")
    return out


def gumbel_fill(seed: int, step: int, rows: int, vocab: int, noise_stream: int = 0,
                device="cuda", stream=None):
    out = torch.empty(rows, vocab, dtype=torch.float32, device=device)
    _check(_lib().ldr_gumbel_fill(int(seed), int(step), int(noise_stream), rows, vocab, _ptr(out),
                                  _stream(stream)), "ldr_gumbel_fill")
    return out


def device_weights(w: Dict, device="cuda") -> Dict:
    """A synth weight dict moved to `device`."""
    out = {k: v.to(device) for k, v in w.items() if k != "layers"}
    out["layers"] = [{k: v.to(device) for k, v in L.items()} for L in w["layers"]]
    return out


def sample_markov(logits: torch.Tensor, anchor: torch.Tensor, E_c: torch.Tensor,
                  W_c: torch.Tensor, temperature: float, top_k: int, seed: int, step: int,
                  out=None, workspace: Optional[torch.Tensor] = None, stream=None):
    """ldr_sample_markov over [batch][B][V] fp32 logits (corrected in place):
    (tokens int32, lse fp32, logq fp32), each [batch][B]."""
    batch, B, V = logits.shape
    rank = E_c.shape[1]
    dtype = LDR_BF16 if E_c.dtype == torch.bfloat16 else LDR_F32
    dev = logits.device
    if out is None:
        out = (torch.empty(batch, B, dtype=torch.int32, device=dev),
               torch.empty(batch, B, dtype=torch.float32, device=dev),
               torch.empty(batch, B, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = torch.empty(sample_workspace_bytes(batch, V), dtype=torch.uint8, device=dev)
    tok, lse, logq = out
    _check(_lib().ldr_sample_markov(_ptr(logits), batch, B, V, _ptr(anchor), _ptr(E_c),
                                    _ptr(W_c), rank, dtype, float(temperature), int(top_k),
                                    int(seed), int(step), _ptr(tok), _ptr(lse), _ptr(logq),
                                    _ptr(workspace), workspace.numel(), _stream(stream)),
           "ldr_sample_markov")
    return tok, lse, logq


def verify_workspace_bytes(batch: int, block: int, vocab: int) -> int:
    return int(_lib().ldr_verify_workspace_bytes(batch, block, vocab))


def verify(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor],
           draft_lse: Optional[torch.Tensor], draft_tokens: torch.Tensor, temperature: float,
           seed: int, step: int, out=None, workspace: Optional[torch.Tensor] = None,
           stream=None, top_k: int = 0):
    """ldr_verify: target logits [batch][B + 1][V], draft logits [batch][B][V]
    with the sampler's lse [batch][B] and tokens [batch][B] (drawn with
    top_k) -> (accepted, next_token, n_new), int32 [batch] each."""
    batch, B1, V = target_logits.shape
    B = B1 - 1
    dev = target_logits.device
    if out is None:
        out = tuple(torch.empty(batch, dtype=torch.int32, device=dev) for _ in range(3))
    if workspace is None:
        workspace = torch.empty(verify_workspace_bytes(batch, B, V), dtype=torch.uint8, device=dev)
    acc, tok, n_new = out
    _check(_lib().ldr_verify(_ptr(target_logits), _ptr(draft_logits), _ptr(draft_lse),
                             _ptr(draft_tokens), batch, B, V, float(temperature), int(top_k),
                             int(seed), int(step), _ptr(acc), _ptr(tok), _ptr(n_new),
                             _ptr(workspace),
                             workspace.numel(), _stream(stream)), "ldr_verify")
    return out


def draft_step_sample_workspace_bytes(shape, batch: int) -> int:
    return int(_lib().ldr_draft_step_sample_workspace_bytes(ctypes.byref(config(shape)), batch))


def draft_step_sample(views: "Views", w: "DraftWeights", anchor: torch.Tensor, temperature: float,
                      seed: int, step: int, logits=True, out=None,
                      workspace: Optional[torch.Tensor] = None, stream=None):
    """ldr_draft_step_sample: (logits or None, tokens, lse, logq); logits=True
    allocates and fills [batch][B][V] fp32 logits, a tensor is filled, None
    asks the fused head not to write them."""
    s, batch = views.shape, views.batch
    dev = anchor.device
    if logits is True:
        logits = torch.empty(batch, s.block, s.vocab, dtype=torch.float32, device=dev)
    if out is None:
        out = (torch.empty(batch, s.block, dtype=torch.int32, device=dev),
               torch.empty(batch, s.block, dtype=torch.float32, device=dev),
               torch.empty(batch, s.block, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = torch.empty(draft_step_sample_workspace_bytes(s, batch), dtype=torch.uint8,
                                device=dev)
    tok, lse, logq = out
    _check(_lib().ldr_draft_step_sample(views.handle, ctypes.byref(w.c), _ptr(anchor), _ptr(logits),
                                        float(temperature), int(seed), int(step), _ptr(tok),
                                        _ptr(lse), _ptr(logq), _ptr(workspace), workspace.numel(),
                                        _stream(stream)), "ldr_draft_step_sample")
    return logits, tok, lse, logq
