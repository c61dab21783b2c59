"""Oracle for the three VLM stages: vision encode, LLM prefill, LLM decode (float64).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Each function is the plain definition
of one step, with no blocking, fusion or reordering, so that it can be checked against the
paper by eye.

What the paper fixes (Sec. 2.1, "GUI-based Agentic VLM"; Sec. 2.2 "VLM Computation Stages"):
  * a ViT encoder turns the screenshot into visual embeddings, a lightweight adapter maps
    them to the LLM width, and the LLM consumes [visual embeddings ; instruction tokens];
  * prefill runs the LLM over that whole sequence and builds the KV cache; decode emits one
    token per step from the cached keys and values (paged blocks, Sec. 1 and Sec. 5.1);
  * decode requests are batched in flight (Sec. 3.4), so a decode step serves B sequences.

Where the paper is silent the readings are (identical on the HIP side):
  pre-LN ViT layer with exact-erf GELU MLP and biased linears; learned absolute position
  embeddings, no class token; patch vector order (row-in-patch, col-in-patch, channel);
  adapter = LayerNorm per patch, concatenation of each 2x2 patch group
  ((2i,2j),(2i,2j+1),(2i+1,2j),(2i+1,2j+1)), one biased Linear (merge=1: LayerNorm + Linear);
  LLM layer = RMSNorm -> Q,K,V (no bias) -> rotary embedding with half-split pairing
  (i, i+d/2) -> causal grouped-query attention (query head h reads KV head h // (n_q/n_kv))
  -> output projection + residual -> RMSNorm -> SwiGLU MLP + residual; final RMSNorm,
  untied LM head, greedy argmax with ties to the lowest index; LayerNorm uses the biased
  variance; RMSNorm is x / sqrt(mean(x^2) + eps) * g.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

F64 = np.float64


# --------------------------------------------------------------------------------------
# elementwise and normalisation steps
# --------------------------------------------------------------------------------------
def layer_norm(x, g, b, eps):
    """LayerNorm over the last axis with biased variance."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(g, F64) + np.asarray(b, F64)


def rms_norm(x, g, eps):
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x, F64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * np.asarray(g, F64)


def gelu(x):
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def softmax(s):
    """Softmax over the last axis (entries of -inf get probability 0)."""
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def linear(x, w, b=None):
    """y = x W^T (+ b) with W stored [out, in]."""
    y = np.asarray(x, F64) @ np.asarray(w, F64).T
    if b is not None:
        y = y + np.asarray(b, F64)
    return y


# --------------------------------------------------------------------------------------
# attention and rotary embedding
# --------------------------------------------------------------------------------------
def attention(q, k, v, causal=False, q_pos=None, k_pos=None):
    """Scaled dot-product attention, one softmax per query row.

    q: [Sq, n_q, d]; k, v: [Sk, n_kv, d].  Query head h reads KV head h // (n_q // n_kv).
    With ``causal``, key j is visible to query i iff k_pos[j] <= q_pos[i].
    Returns [Sq, n_q, d].
    """
    q, k, v = (np.asarray(t, F64) for t in (q, k, v))
    sq, nq, d = q.shape
    nkv = k.shape[1]
    group = nq // nkv
    out = np.empty((sq, nq, v.shape[2]), F64)
    for h in range(nq):
        g = h // group
        s = q[:, h, :] @ k[:, g, :].T / math.sqrt(d)
        if causal:
            visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
            s = np.where(visible, s, -np.inf)
        out[:, h, :] = softmax(s) @ v[:, g, :]
    return out


def rope(x, pos, theta):
    """Rotary position embedding, half-split pairing: dims (i, i + d/2) rotate by pos * theta^(-2i/d).

    x: [S, heads, d]; pos: [S] integer positions.
    """
    x = np.asarray(x, F64)
    d = x.shape[-1]
    half = d // 2
    inv_freq = float(theta) ** (-np.arange(half, dtype=F64) * 2.0 / d)
    ang = np.asarray(pos, F64)[:, None] * inv_freq[None, :]          # [S, half]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


# --------------------------------------------------------------------------------------
# vision encode (ViT + adapter)
# --------------------------------------------------------------------------------------
def patchify(img, p):
    """[H, W, C] image -> [N, p*p*C] patches, row-major over the patch grid, vector order (py, px, c)."""
    img = np.asarray(img, F64)
    h, w, c = img.shape
    gh, gw = h // p, w // p
    x = img[:gh * p, :gw * p].reshape(gh, p, gw, p, c).transpose(0, 2, 1, 3, 4)
    return x.reshape(gh * gw, p * p * c)


def patch_embed(img, w, cfg):
    """x0 = patches W_p^T + b_p + E_pos."""
    return linear(patchify(img, cfg.patch), w["patch.w"], w["patch.b"]) + np.asarray(w["pos"], F64)


def vit_layer(x, w, l, cfg, rows=None):
    """One pre-LN encoder layer with bidirectional attention over all patches.

    h = x + Attn(LN1(x)) W_o^T + b_o ;  y = h + GELU(LN2(h) W_1^T + b_1) W_2^T + b_2.
    ``rows`` restricts the output to those query rows (keys and values still span all patches).
    """
    p = f"l{l}."
    x = np.asarray(x, F64)
    n, hid = x.shape
    nh, d = cfg.heads, cfg.hidden // cfg.heads
    a = layer_norm(x, w[p + "ln1.g"], w[p + "ln1.b"], cfg.eps)
    qkv = linear(a, w[p + "qkv.w"], w[p + "qkv.b"])
    q = qkv[:, :hid].reshape(n, nh, d)
    k = qkv[:, hid:2 * hid].reshape(n, nh, d)
    v = qkv[:, 2 * hid:].reshape(n, nh, d)
    if rows is not None:
        q, x = q[rows], x[rows]
    att = attention(q, k, v, causal=False)
    h = x + linear(att.reshape(att.shape[0], hid), w[p + "o.w"], w[p + "o.b"])
    m = gelu(linear(layer_norm(h, w[p + "ln2.g"], w[p + "ln2.b"], cfg.eps), w[p + "fc1.w"], w[p + "fc1.b"]))
    return h + linear(m, w[p + "fc2.w"], w[p + "fc2.b"])


def merge_adapter(x, w, cfg):
    """Adapter from ViT width to LLM width.

    merge == 1: LN + Linear per patch.  merge == 2: LN per patch, concatenate each 2x2 patch
    group in the order (2i,2j), (2i,2j+1), (2i+1,2j), (2i+1,2j+1), then one Linear; merged
    tokens are row-major over the (gh/2, gw/2) grid.
    """
    hid = cfg.hidden
    a = layer_norm(x, w["merge.ln.g"], w["merge.ln.b"], cfg.eps)
    m = cfg.merge
    if m > 1:
        gh, gw = cfg.grid_h, cfg.grid_w
        a = a.reshape(gh // m, m, gw // m, m, hid).transpose(0, 2, 1, 3, 4).reshape(gh * gw // (m * m), m * m * hid)
    return linear(a, w["merge.w"], w["merge.b"])


def vit_encode(img, w, cfg, layers=None):
    """Vision encode of one image [H, W, C] -> [n_out, out_hidden] LLM-width embeddings."""
    x = patch_embed(img, w, cfg)
    for l in range(cfg.layers if layers is None else layers):
        x = vit_layer(x, w, l, cfg)
    return merge_adapter(x, w, cfg)


def vit_encode_tokens(img, w, cfg, tokens):
    """Vision encode evaluated only at the merged output ``tokens`` (row-major over the merged grid).

    Every layer but the last runs on all patches; the last one only at the patches the
    requested tokens merge ((2i,2j), (2i,2j+1), (2i+1,2j), (2i+1,2j+1) for token (i, j)), with
    keys and values from all patches.  Returns [len(tokens), out_hidden].
    """
    x = patch_embed(img, w, cfg)
    for l in range(cfg.layers - 1):
        x = vit_layer(x, w, l, cfg)
    m, gw = cfg.merge, cfg.grid_w
    rows = []
    for t in tokens:
        i, j = divmod(int(t), gw // m)
        rows += [(m * i + dy) * gw + (m * j + dx) for dy in range(m) for dx in range(m)]
    y = vit_layer(x, w, cfg.layers - 1, cfg, rows=np.array(rows)) if cfg.layers > 0 else x[np.array(rows)]
    a = layer_norm(y, w["merge.ln.g"], w["merge.ln.b"], cfg.eps).reshape(len(tokens), m * m * cfg.hidden)
    return linear(a, w["merge.w"], w["merge.b"])


# --------------------------------------------------------------------------------------
# paged KV cache
# --------------------------------------------------------------------------------------
class PagedKV:
    """KV cache in fixed-size blocks (PagedAttention style): K[layer][block][kv_head][slot][d]."""

    def __init__(self, layers, num_blocks, n_kv, block, d):
        self.block = block
        self.k = np.zeros((layers, num_blocks, n_kv, block, d), F64)
        self.v = np.zeros((layers, num_blocks, n_kv, block, d), F64)

    def write(self, l, table, pos, k, v):
        """Store k, v ([n, n_kv, d]) for positions ``pos`` of the sequence whose block table is ``table``."""
        for i, p in enumerate(np.asarray(pos)):
            blk = int(table[p // self.block])
            self.k[l, blk, :, p % self.block, :] = k[i]
            self.v[l, blk, :, p % self.block, :] = v[i]

    def read(self, l, table, n):
        """Keys and values of positions 0..n-1 as contiguous [n, n_kv, d] arrays."""
        ks, vs = [], []
        for p in range(n):
            blk = int(table[p // self.block])
            ks.append(self.k[l, blk, :, p % self.block, :])
            vs.append(self.v[l, blk, :, p % self.block, :])
        return np.stack(ks), np.stack(vs)


# --------------------------------------------------------------------------------------
# LLM prefill and decode
# --------------------------------------------------------------------------------------
def bf16_store(x):
    """A tensor as a bf16 model stores it: each value rounded to the nearest bfloat16 (ties to
    even), returned as float64.  The paper runs its models in bf16 (Sec. 5.1), so the activations
    a bf16 model keeps between operations and its KV cache hold bf16 values.  Values are taken to
    float32 first (the precision the arithmetic between two stores works in), then rounded.
    """
    f = np.ascontiguousarray(np.asarray(x, F64), dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    out = r.astype(np.uint32).view(np.float32).astype(F64)
    return np.where(np.isnan(f), np.nan, out)


def _keep(x):
    return x


def _qkv(h, w, l, cfg, pos, store=_keep):
    p = f"l{l}."
    n = h.shape[0]
    d = cfg.head_dim
    q = store(rope(store(linear(h, w[p + "q.w"])).reshape(n, cfg.n_q, d), pos, cfg.rope_theta))
    k = store(rope(store(linear(h, w[p + "k.w"])).reshape(n, cfg.n_kv, d), pos, cfg.rope_theta))
    v = store(linear(h, w[p + "v.w"])).reshape(n, cfg.n_kv, d)
    return q, k, v


def _mlp(x, w, l, cfg, store=_keep):
    p = f"l{l}."
    h = store(rms_norm(x, w[p + "rms2.g"], cfg.eps))
    return linear(store(silu(linear(h, w[p + "gate.w"])) * linear(h, w[p + "up.w"])), w[p + "down.w"])


def lm_head(x, w, cfg, store=_keep):
    """Final RMSNorm and untied LM head: [n, H] -> [n, vocab] logits."""
    return linear(store(rms_norm(x, w["norm.g"], cfg.eps)), w["lm_head.w"])


def greedy(logits):
    """Greedy next token: argmax over the vocabulary, ties to the lowest index."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.int32)


def llm_prefill(vis, ids, w, cfg, kv=None, table=None, return_hidden=False, store=_keep):
    """Prefill one request over [visual embeddings ; embedded instruction tokens].

    Causal attention spans the whole concatenated sequence; positions are 0..S-1.  If a
    paged cache is given, every layer's rotated K and V are written through ``table``.
    Returns (last-row logits [vocab], next token id) and optionally the final hidden states.

    ``store`` is applied to every tensor a model keeps between operations: the normed input
    of each projection, the q / k / v projections, the rotated q and k, the attention output,
    the MLP hidden activation and the final normed row (the residual stream is kept as is).
    The default keeps exact values; ``bf16_store`` evaluates the same definition as a bf16
    model stores its tensors.
    """
    vis = np.asarray(vis, F64).reshape(-1, cfg.hidden)
    x = np.concatenate([vis, np.asarray(w["embed"], F64)[np.asarray(ids)]], axis=0)
    s = x.shape[0]
    pos = np.arange(s)
    for l in range(cfg.layers):
        p = f"l{l}."
        q, k, v = _qkv(store(rms_norm(x, w[p + "rms1.g"], cfg.eps)), w, l, cfg, pos, store)
        if kv is not None:
            kv.write(l, table, pos, k, v)
        att = store(attention(q, k, v, causal=True, q_pos=pos, k_pos=pos))
        x = x + linear(att.reshape(s, cfg.n_q * cfg.head_dim), w[p + "o.w"])
        x = x + _mlp(x, w, l, cfg, store)
    logits = lm_head(x[-1:], w, cfg, store)[0]
    if return_hidden:
        return logits, int(greedy(logits)), x
    return logits, int(greedy(logits))


def llm_decode_step(ids, pos, tables, kv, w, cfg, store=_keep):
    """One in-flight-batched decode step.

    Sequence b feeds token ids[b] at position pos[b]: its K, V are appended to the paged
    cache, and its single query attends to cached positions 0..pos[b].
    Returns (logits [B, vocab], next ids [B]).  ``store`` as in llm_prefill.
    """
    ids = np.asarray(ids)
    pos = np.asarray(pos)
    bsz = ids.shape[0]
    x = np.asarray(w["embed"], F64)[ids]
    for l in range(cfg.layers):
        p = f"l{l}."
        h = store(rms_norm(x, w[p + "rms1.g"], cfg.eps))
        att = np.empty((bsz, cfg.n_q, cfg.head_dim), F64)
        for b in range(bsz):
            q, k, v = _qkv(h[b:b + 1], w, l, cfg, pos[b:b + 1], store)
            kv.write(l, tables[b], pos[b:b + 1], k, v)
            kc, vc = kv.read(l, tables[b], int(pos[b]) + 1)
            att[b] = attention(q, kc, vc, causal=False)[0]
        x = x + linear(store(att).reshape(bsz, cfg.n_q * cfg.head_dim), w[p + "o.w"])
        x = x + _mlp(x, w, l, cfg, store)
    logits = lm_head(x, w, cfg, store)
    return logits, greedy(logits)


def llm_layer_rows(x, w, l, cfg, rows):
    """One prefill layer (positions 0..S-1) evaluated only at query ``rows``.

    K and V come from every position; used to check sampled rows of a full-width layer.
    Returns (layer output at ``rows`` [len(rows), H], rotated K [S, n_kv, d], V [S, n_kv, d]).
    """
    p = f"l{l}."
    x = np.asarray(x, F64)
    s = x.shape[0]
    pos = np.arange(s)
    q, k, v = _qkv(rms_norm(x, w[p + "rms1.g"], cfg.eps), w, l, cfg, pos)
    rows = np.asarray(rows)
    att = attention(q[rows], k, v, causal=True, q_pos=pos[rows], k_pos=pos)
    h = x[rows] + linear(att.reshape(len(rows), cfg.n_q * cfg.head_dim), w[p + "o.w"])
    return h + _mlp(h, w, l, cfg), k, v


# --------------------------------------------------------------------------------------
# comparison metric
# --------------------------------------------------------------------------------------
def max_rel_err(got, ref):
    """Norm-wise relative error max|got - ref| / max|ref| over one output tensor."""
    got = np.asarray(got, F64)
    ref = np.asarray(ref, F64)
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))
