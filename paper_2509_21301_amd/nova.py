"""Python binding of libnova (ctypes).  Argument marshalling only: every step of the three stages
runs in the HIP kernels behind the C ABI declared in ``include/nova.h``.

PyTorch provides device memory, pinned host memory and streams.  The library must be built
(``python -m paper_2509_21301_amd.build``); importing this module without it raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnova.so")

OK, EINVAL, ENOKV, EHIP, EUNSUPPORTED, ENOSPACE = 0, -1, -2, -3, -4, -5
STAGE_ENCODE, STAGE_PREFILL, STAGE_DECODE = 0, 1, 2
ACT_BF16, ACT_F32 = 0, 1
KIND_GEMM, KIND_ATTN, KIND_GEMV, KIND_DECODE_ATTN, KIND_MISC = 0, 1, 2, 3, 4
KIND_NAMES = {KIND_GEMM: "gemm", KIND_ATTN: "attention", KIND_GEMV: "thin_gemm", KIND_DECODE_ATTN: "decode_attention",
              KIND_MISC: "misc"}


class NovaError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libnova error {code}: {msg}")
        self.code = code


class VitConfigC(C.Structure):
    _fields_ = [("hidden", C.c_int), ("heads", C.c_int), ("mlp", C.c_int), ("layers", C.c_int), ("patch", C.c_int),
                ("merge", C.c_int), ("out_hidden", C.c_int), ("image_h", C.c_int), ("image_w", C.c_int),
                ("eps", C.c_float), ("act", C.c_int)]


class VitDescC(C.Structure):
    _fields_ = [("cfg", VitConfigC), ("embed", C.c_void_p), ("head", C.c_void_p), ("layers", C.c_void_p),
                ("host_layers", C.c_void_p), ("slots", C.c_void_p), ("n_slots", C.c_int)]


class LlmConfigC(C.Structure):
    _fields_ = [("hidden", C.c_int), ("n_q", C.c_int), ("n_kv", C.c_int), ("head_dim", C.c_int), ("inter", C.c_int),
                ("vocab", C.c_int), ("layers", C.c_int), ("block", C.c_int), ("rope_theta", C.c_float),
                ("eps", C.c_float), ("act", C.c_int)]


class LlmDescC(C.Structure):
    _fields_ = [("cfg", LlmConfigC), ("embed", C.c_void_p), ("layers", C.c_void_p), ("head", C.c_void_p)]


class KvC(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("num_blocks", C.c_int)]


# symbol -> (restype, argtypes); mirrors include/nova.h
_SIG = {
    "nova_last_error": (C.c_char_p, []),
    "nova_init": (C.c_int, [C.c_int]),
    "nova_shutdown": (None, []),
    "nova_device_cus": (C.c_int, []),
    "nova_vit_embed_layout": (C.c_int, [C.POINTER(VitConfigC), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "nova_vit_layer_layout": (C.c_int, [C.POINTER(VitConfigC), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "nova_vit_head_layout": (C.c_int, [C.POINTER(VitConfigC), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "nova_vit_create": (C.c_int, [C.POINTER(VitDescC), C.POINTER(C.c_void_p)]),
    "nova_vit_destroy": (None, [C.c_void_p]),
    "nova_vit_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int]),
    "nova_vit_encode": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "nova_prefetch_layer": (C.c_int, [C.c_void_p, C.c_int, C.c_void_p]),
    "nova_vit_offload_state": (C.c_int, [C.c_void_p, C.POINTER(C.c_int), C.POINTER(C.c_ulonglong)]),
    "nova_llm_layer_layout": (C.c_int, [C.POINTER(LlmConfigC), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "nova_llm_head_layout": (C.c_int, [C.POINTER(LlmConfigC), C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "nova_llm_create": (C.c_int, [C.POINTER(LlmDescC), C.POINTER(C.c_void_p)]),
    "nova_llm_destroy": (None, [C.c_void_p]),
    "nova_kv_bytes": (C.c_size_t, [C.c_void_p, C.c_int]),
    "nova_llm_prefill_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int]),
    "nova_llm_decode_workspace_bytes": (C.c_size_t, [C.c_void_p, C.c_int, C.c_int]),
    "nova_llm_prefill": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_int, C.c_void_p, C.POINTER(KvC),
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "nova_llm_decode": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_int,
                                  C.POINTER(KvC), C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "nova_llm_decode_noalloc": (C.c_int, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_int,
                                          C.POINTER(KvC), C.c_void_p, C.c_void_p, C.c_void_p]),
    "nova_linear": (C.c_int, [C.c_int, C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p]),
    "nova_make_cu_mask": (C.c_int, [C.c_int, C.c_int, C.POINTER(C.c_uint32)]),
    "nova_set_stage_partition": (C.c_int, [C.c_int, C.POINTER(C.c_uint32), C.c_int, C.POINTER(C.c_void_p)]),
    "nova_cu_probe": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int]),
    "nova_timing_enable": (C.c_int, [C.c_int]),
    "nova_timing_read": (C.c_int, [C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_int)]),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2509_21301_amd.build`")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in _SIG.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()


def _check(rc):
    if rc != OK:
        raise NovaError(rc, lib.nova_last_error().decode())
    return rc


def init(device: int = 0):
    _check(lib.nova_init(device))


def device_cus() -> int:
    return lib.nova_device_cus()


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# ----------------------------------------------------------------------------- layouts
def _layout(fn, cfg, n):
    off = (C.c_size_t * n)()
    size = C.c_size_t()
    _check(fn(C.byref(cfg), off, C.byref(size)))
    return list(off), size.value


def vit_config_c(cfg, act=ACT_BF16) -> VitConfigC:
    return VitConfigC(cfg.hidden, cfg.heads, cfg.mlp, cfg.layers, cfg.patch, cfg.merge, cfg.out_hidden, cfg.image_h,
                      cfg.image_w, cfg.eps, act)


def llm_config_c(cfg, act=ACT_BF16) -> LlmConfigC:
    return LlmConfigC(cfg.hidden, cfg.n_q, cfg.n_kv, cfg.head_dim, cfg.inter, cfg.vocab, cfg.layers, cfg.block,
                      cfg.rope_theta, cfg.eps, act)


def vit_layouts(cfg, act=ACT_BF16):
    c = vit_config_c(cfg, act)
    return (_layout(lib.nova_vit_embed_layout, c, 3), _layout(lib.nova_vit_layer_layout, c, 12),
            _layout(lib.nova_vit_head_layout, c, 4))


def llm_layouts(cfg, act=ACT_BF16):
    c = llm_config_c(cfg, act)
    return _layout(lib.nova_llm_layer_layout, c, 6), _layout(lib.nova_llm_head_layout, c, 2)


def _round(x, m):
    return (x + m - 1) // m * m


# ----------------------------------------------------------------------------- weight packing
def _bf16(a, device) -> torch.Tensor:
    """bf16 copy of a bf16-exact float array (numpy or torch)."""
    t = torch.from_numpy(np.ascontiguousarray(a)) if isinstance(a, np.ndarray) else a
    return t.to(device=device, dtype=torch.bfloat16)


class _Blob:
    def __init__(self, nbytes, device, pin=False):
        if pin:
            self.t = torch.zeros(nbytes // 2, dtype=torch.bfloat16, pin_memory=True)
        else:
            self.t = torch.zeros(nbytes // 2, dtype=torch.bfloat16, device=device)

    def view(self, off, shape):
        n = int(np.prod(shape))
        return self.t[off // 2: off // 2 + n].view(*shape)


def _put(blob, off, src, shape, device):
    """Copy src (rows x cols) into the top-left corner of a zero region of `shape`."""
    v = blob.view(off, shape)
    s = _bf16(src, v.device)
    if s.dim() == 1:
        v[: s.shape[0]].copy_(s)
    else:
        v[: s.shape[0], : s.shape[1]].copy_(s)


def pack_vit(cfg, w, act=ACT_BF16, device="cuda", layer_range=None, pin_layers=False):
    """Pack ViT weights (dict name -> array, as synth.vit_weights gives) into the three blob kinds.

    Returns (embed blob, list-of-layers blob (all layers back to back), head blob) as bf16 tensors.
    """
    (eo, eb), (lo, lb), (ho, hb) = vit_layouts(cfg, act)
    H, I, P = cfg.hidden, _round(cfg.mlp, 256), _round(cfg.patch_dim, 64)
    emb = _Blob(eb, device)
    _put(emb, eo[0], w["patch.w"], (H, P), device)
    _put(emb, eo[1], w["patch.b"], (H,), device)
    _put(emb, eo[2], w["pos"], (cfg.n_patches, H), device)
    layers = list(range(cfg.layers)) if layer_range is None else list(layer_range)
    lay = _Blob(lb * len(layers), device, pin=pin_layers)
    for i, l in enumerate(layers):
        p = f"l{l}."
        base = i * lb
        specs = [("ln1.g", (H,)), ("ln1.b", (H,)), ("qkv.w", (3 * H, H)), ("qkv.b", (3 * H,)), ("o.w", (H, H)),
                 ("o.b", (H,)), ("ln2.g", (H,)), ("ln2.b", (H,)), ("fc1.w", (I, H)), ("fc1.b", (I,)),
                 ("fc2.w", (H, I)), ("fc2.b", (H,))]
        for j, (nm, shp) in enumerate(specs):
            _put(lay, base + lo[j], w[p + nm], shp, device)
    head = _Blob(hb, device)
    m2 = cfg.merge * cfg.merge
    _put(head, ho[0], w["merge.ln.g"], (H,), device)
    _put(head, ho[1], w["merge.ln.b"], (H,), device)
    _put(head, ho[2], w["merge.w"], (cfg.out_hidden, m2 * H), device)
    _put(head, ho[3], w["merge.b"], (cfg.out_hidden,), device)
    return emb.t, lay.t, head.t, lb


def pack_llm(cfg, w, act=ACT_BF16, device="cuda"):
    """Pack LLM weights into (embed table, layers blob, head blob)."""
    (lo, lb), (ho, hb) = llm_layouts(cfg, act)
    H, I, d = cfg.hidden, _round(cfg.inter, 256), cfg.head_dim
    lay = _Blob(lb * cfg.layers, device)
    for l in range(cfg.layers):
        p, base = f"l{l}.", l * lb
        _put(lay, base + lo[0], w[p + "rms1.g"], (H,), device)
        qkv = np.concatenate([w[p + "q.w"], w[p + "k.w"], w[p + "v.w"]], 0) if isinstance(w[p + "q.w"], np.ndarray) \
            else torch.cat([w[p + "q.w"], w[p + "k.w"], w[p + "v.w"]], 0)
        _put(lay, base + lo[1], qkv, ((cfg.n_q + 2 * cfg.n_kv) * d, H), device)
        _put(lay, base + lo[2], w[p + "o.w"], (H, cfg.n_q * d), device)
        _put(lay, base + lo[3], w[p + "rms2.g"], (H,), device)
        gu = lay.view(base + lo[4], (I // 8, 2, 8, H))
        gate = torch.zeros(I, H, dtype=torch.bfloat16, device=gu.device)
        up = torch.zeros(I, H, dtype=torch.bfloat16, device=gu.device)
        gate[: cfg.inter] = _bf16(w[p + "gate.w"], gu.device)
        up[: cfg.inter] = _bf16(w[p + "up.w"], gu.device)
        gu[:, 0].copy_(gate.view(I // 8, 8, H))
        gu[:, 1].copy_(up.view(I // 8, 8, H))
        _put(lay, base + lo[5], w[p + "down.w"], (H, I), device)
    head = _Blob(hb, device)
    _put(head, ho[0], w["norm.g"], (H,), device)
    _put(head, ho[1], w["lm_head.w"], (cfg.vocab, H), device)
    embed = _bf16(w["embed"], device).contiguous()
    return embed, lay.t, head.t, lb


def act_dtype(act):
    return torch.float32 if act == ACT_F32 else torch.bfloat16


# ----------------------------------------------------------------------------- models
class Vit:
    """Vision encoder handle.  With n_slots > 0 the layers stay in pinned host memory and are
    streamed through n_slots device slots."""

    def __init__(self, cfg, weights, act=ACT_BF16, device="cuda", n_slots=0, blobs=None):
        self.cfg, self.act, self.device = cfg, act, device
        if blobs is None:
            blobs = pack_vit(cfg, weights, act, device, pin_layers=n_slots > 0)
        self.embed, self.layers, self.head, self.layer_bytes = blobs
        self.slots = None
        desc = VitDescC(vit_config_c(cfg, act), _ptr(self.embed), _ptr(self.head), None, None, None, 0)
        if n_slots > 0:
            if self.layers.is_cuda:
                raise ValueError("offload needs the layer blob in pinned host memory")
            self.slots = torch.zeros(n_slots * self.layer_bytes // 2, dtype=torch.bfloat16, device=device)
            desc.host_layers = _ptr(self.layers)
            desc.slots = _ptr(self.slots)
            desc.n_slots = n_slots
            self.slots_n = n_slots
        else:
            desc.layers = _ptr(self.layers)
        h = C.c_void_p()
        _check(lib.nova_vit_create(C.byref(desc), C.byref(h)))
        self.h = h
        self._ws = {}

    def workspace(self, batch):
        if batch not in self._ws:
            n = lib.nova_vit_workspace_bytes(self.h, batch)
            self._ws[batch] = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self._ws[batch]

    def out_shape(self, batch):
        return (batch, self.cfg.n_out, self.cfg.out_hidden)

    def encode(self, pixels, out=None, stream=None):
        """pixels: bf16 [B, H, W, 3] on the device -> act-type [B, n_out, out_hidden]."""
        assert pixels.dtype == torch.bfloat16 and pixels.is_cuda and pixels.is_contiguous()
        b = pixels.shape[0]
        if out is None:
            out = torch.empty(self.out_shape(b), dtype=act_dtype(self.act), device=self.device)
        ws = self.workspace(b)
        _check(lib.nova_vit_encode(self.h, _ptr(pixels), b, _ptr(out), _ptr(ws), ws.numel(), _stream(stream)))
        return out

    def prefetch(self, layer, stream=None):
        _check(lib.nova_prefetch_layer(self.h, layer, None if stream is None else stream.cuda_stream))

    def offload_state(self):
        """(logical layer held by each physical slot, layer copies issued so far)."""
        k = C.c_int * self.slots_n
        sl, n = k(), C.c_ulonglong()
        _check(lib.nova_vit_offload_state(self.h, sl, C.byref(n)))
        return list(sl), n.value

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value and lib is not None:
            lib.nova_vit_destroy(h)
            self.h = None


class KvPool:
    def __init__(self, llm, num_blocks, device="cuda"):
        n = lib.nova_kv_bytes(llm.h, num_blocks)
        dt = act_dtype(llm.act)
        el = n // torch.tensor([], dtype=dt).element_size()
        self.k = torch.zeros(el, dtype=dt, device=device)
        self.v = torch.zeros(el, dtype=dt, device=device)
        self.num_blocks = num_blocks
        self.c = KvC(_ptr(self.k), _ptr(self.v), num_blocks)
        cfg = llm.cfg
        self.k5 = self.k.view(cfg.layers, num_blocks, cfg.n_kv, cfg.block, cfg.head_dim)
        self.v5 = self.v.view(cfg.layers, num_blocks, cfg.n_kv, cfg.head_dim, cfg.block)


class Llm:
    def __init__(self, cfg, weights, act=ACT_BF16, device="cuda", blobs=None):
        self.cfg, self.act, self.device = cfg, act, device
        if blobs is None:
            blobs = pack_llm(cfg, weights, act, device)
        self.embed, self.layers, self.head, self.layer_bytes = blobs
        desc = LlmDescC(llm_config_c(cfg, act), _ptr(self.embed), _ptr(self.layers), _ptr(self.head))
        h = C.c_void_p()
        _check(lib.nova_llm_create(C.byref(desc), C.byref(h)))
        self.h = h
        self._ws = {}
        self._retired = []

    def _workspace(self, key, nbytes, stream=None):
        t = self._ws.get(key)
        if t is None or t.numel() < nbytes:
            if t is not None:
                # the old buffer may still be read by work queued earlier by this stage; keep it
                # until an event recorded now on this call's stream has completed (the library
                # orders a stage's new partition stream after its earlier ones), so the caching
                # allocator cannot hand it out while the GPU still uses it
                ev = torch.cuda.Event()
                ev.record(stream if stream is not None else torch.cuda.current_stream())
                self._retired.append((t, ev))
            t = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
            self._ws[key] = t
        if self._retired:
            self._retired = [(b, e) for b, e in self._retired if not e.query()]
        return t

    def reserve(self, prefill_tokens=0, decode_batch=0, decode_ctx=0):
        """Size the prefill and decode workspaces once for the largest calls to come, so that no
        later call grows them (a serving worker then never waits on a buffer swap)."""
        if prefill_tokens > 0:
            self._workspace("prefill", lib.nova_llm_prefill_workspace_bytes(self.h, prefill_tokens))
        if decode_batch > 0 and decode_ctx > 0:
            # the attention split count falls with the batch, so the largest need is not always at
            # the largest batch
            need = max(lib.nova_llm_decode_workspace_bytes(self.h, b, decode_ctx) for b in range(1, decode_batch + 1))
            self._workspace("decode", need)

    def prefill(self, vis, ids, table, kv, logits=None, next_id=None, stream=None):
        n_vis = 0 if vis is None else vis.shape[0]
        n_text = ids.shape[0]
        ws = self._workspace("prefill", lib.nova_llm_prefill_workspace_bytes(self.h, n_vis + n_text), stream)
        if next_id is None:
            next_id = torch.empty(1, dtype=torch.int32, device=self.device)
        _check(lib.nova_llm_prefill(self.h, _ptr(vis), n_vis, _ptr(ids), n_text, _ptr(table), C.byref(kv.c),
                                    _ptr(next_id), _ptr(logits), _ptr(ws), ws.numel(), _stream(stream)))
        return next_id

    def decode(self, ids, pos, tables, kv, max_ctx, next_ids=None, logits=None, stream=None):
        b = ids.shape[0]
        # one decode workspace for every batch size: a larger one serves a smaller step as well
        ws = self._workspace("decode", lib.nova_llm_decode_workspace_bytes(self.h, b, max_ctx), stream)
        if next_ids is None:
            next_ids = torch.empty(b, dtype=torch.int32, device=self.device)
        _check(lib.nova_llm_decode(self.h, _ptr(ids), _ptr(pos), _ptr(tables), tables.shape[1], b, max_ctx,
                                   C.byref(kv.c), _ptr(next_ids), _ptr(logits), _ptr(ws), ws.numel(),
                                   _stream(stream)))
        return next_ids

    def decode_noalloc(self, ids, pos, tables, kv, max_ctx, next_ids, logits=None, stream=None):
        """The same step with the library's static scratch as workspace (no allocation in the
        library; outputs are the caller's)."""
        _check(lib.nova_llm_decode_noalloc(self.h, _ptr(ids), _ptr(pos), _ptr(tables), tables.shape[1], ids.shape[0],
                                           max_ctx, C.byref(kv.c), _ptr(next_ids), _ptr(logits), _stream(stream)))
        return next_ids

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value and lib is not None:
            lib.nova_llm_destroy(h)
            self.h = None


# ----------------------------------------------------------------------------- linear co-run study
LINEAR_TILED, LINEAR_TILED_SMALL, LINEAR_THIN, LINEAR_THIN_VALU = 0, 1, 2, 3


def linear(variant: int, x, w, out, stream=None):
    """out (fp32 [M, N]) += x (bf16 [M, K]) w (bf16 [N, K])^T with the chosen kernel variant."""
    m, k = x.shape
    n = w.shape[0]
    _check(lib.nova_linear(variant, _ptr(x), m, k, _ptr(w), n, _ptr(out), _stream(stream)))
    return out


# ----------------------------------------------------------------------------- partitions & timing
def make_cu_mask(n_cus: int, first_slot: int = 0) -> list[int]:
    m = (C.c_uint32 * 8)()
    _check(lib.nova_make_cu_mask(n_cus, first_slot, m))
    return list(m)


def set_stage_partition(stage: int, mask) -> torch.cuda.ExternalStream:
    arr = (C.c_uint32 * len(mask))(*mask)
    s = C.c_void_p()
    _check(lib.nova_set_stage_partition(stage, arr, len(mask), C.byref(s)))
    return torch.cuda.ExternalStream(s.value)


def cu_probe(stream, n_workgroups: int = 4096):
    """(xcd, shader engine, cu) of the CU each probe workgroup ran on, as a set."""
    out = torch.zeros(n_workgroups, dtype=torch.int32, device="cuda")
    _check(lib.nova_cu_probe(_stream(stream), _ptr(out), n_workgroups))
    stream = stream or torch.cuda.current_stream()
    stream.synchronize()
    v = out.cpu().numpy().astype(np.uint32)
    return {(int(x >> 16), int((x >> 8) & 0xff), int(x & 0xff)) for x in v}


def timing_enable(on: bool = True):
    _check(lib.nova_timing_enable(1 if on else 0))


def timing_read(kind: int):
    ms = C.c_double()
    n = C.c_int()
    _check(lib.nova_timing_read(kind, C.byref(ms), C.byref(n)))
    return ms.value, n.value
