"""Plain numpy decoder: the definition the stage engine must reproduce.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed, and where the paper says so:

* Section 2.1 (LLM Inference): a prompt is processed in one prefill pass that
  produces the first token and stores every token's key and value vectors;
  each decode step then reuses that cache and produces one more token.
* Section 2.1 and section 4.1 (tradeoff analysis): pipeline parallelism gives
  each worker a contiguous range of layers and passes intermediate results
  from worker to worker in order; for Llama2-7B that intermediate result is
  8 KB per token, i.e. one 16-bit hidden vector of 4096 values.
* Section 6 and 6.2: after consolidation one worker runs the whole model; the
  KV blocks it receives are placed at the layers of the worker they came
  from. Migration therefore moves cache content without changing it.

The paper names the model family (Llama2, section 8 setup) but does not spell
out the layer. The readings used here are the standard Llama ones: pre-norm
RMSNorm, rotate-half rotary embedding on q and k, causal softmax attention
with scale 1/sqrt(d) and grouped KV heads (query head h reads KV head
h // (n_heads / n_kv_heads)), SwiGLU feed-forward, no biases, untied LM head.

Every array is float32 unless ``dtype=np.float64`` is requested. Sequences
are processed one at a time with whole-matrix numpy operations; nothing is
blocked, fused or reordered.
"""
from __future__ import annotations

import numpy as np

from workloads import gen as _gen


# ---------------------------------------------------------------- primitives

def rms_norm(x, g, eps):
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + x.dtype.type(eps)) * g


def rope_angles(positions, head_dim, base):
    """cos and sin of pos * base^(-2i/d) for i < d/2, computed in float64.

    Rotate-half convention: element i is paired with element i + d/2."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(np.float64(base), -2.0 * i / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x, cos, sin):
    """Rotate x [T, n_heads, d] by the per-position angles (cos/sin [T, d/2])."""
    half = x.shape[-1] // 2
    c = cos.astype(x.dtype)[:, None, :]
    s = sin.astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention_probs(q, k, q_pos, k_pos, scale):
    """Causal softmax(q k^T * scale) for one head: q [Tq, d], k [Tk, d].

    Key j is visible to query i iff k_pos[j] <= q_pos[i]."""
    s = (q @ k.T) * q.dtype.type(scale)
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    s = np.where(visible, s, -np.inf)
    s = s - np.max(s, axis=1, keepdims=True)
    p = np.exp(s)
    return p / np.sum(p, axis=1, keepdims=True)


def attention(q, k, v, q_pos, k_pos):
    """Grouped-query causal attention.

    q [Tq, n_heads, d]; k, v [Tk, n_kv_heads, d] -> [Tq, n_heads * d]."""
    n_heads, d = q.shape[1], q.shape[2]
    n_rep = n_heads // k.shape[1]
    scale = 1.0 / np.sqrt(np.float64(d))
    out = np.empty((q.shape[0], n_heads, d), dtype=q.dtype)
    for h in range(n_heads):
        kh = h // n_rep
        p = attention_probs(q[:, h], k[:, kh], q_pos, k_pos, scale)
        out[:, h] = p @ v[:, kh]
    return out.reshape(q.shape[0], n_heads * d)


def silu(z):
    return z / (z.dtype.type(1) + np.exp(-z))


def swiglu(u, wg, wu, wd):
    """(silu(u wg^T) * (u wu^T)) wd^T."""
    return (silu(u @ wg.T) * (u @ wu.T)) @ wd.T


def argmax_lowest(logits):
    """Greedy choice: index of the maximum, the lowest index among ties
    (numpy's argmax returns the first occurrence)."""
    return np.argmax(logits, axis=-1).astype(np.int32)


# ------------------------------------------------------------------- weights

class SyntheticWeights:
    """Weight source for the oracle: the seeded draws of ``workloads.gen``.

    ``bf16=True`` rounds each draw to bfloat16 first (diagnostic mode that
    separates weight rounding from kernel error). ``keep`` caches the arrays;
    turn it off for models too big to hold in float32.
    """

    def __init__(self, cfg, bf16=False, keep=True):
        self.cfg, self.bf16, self.keep = cfg, bf16, keep
        self._cache = {}

    def __call__(self, layer, kind):
        key = (layer, kind)
        if key in self._cache:
            return self._cache[key]
        if kind in ("attn_norm", "ffn_norm", "final_norm"):
            w = _gen.gains(self.cfg)
        else:
            w = _gen.weight_f32(self.cfg, layer, kind)
            if self.bf16:
                w = _gen.round_to_bf16(w)
        if self.keep:
            self._cache[key] = w
        return w


# --------------------------------------------------------------------- stage

class Stage:
    """One pipeline stage: layers [begin, end) of the model.

    The first stage (begin == 0) takes token ids and looks up the
    embedding; the last stage (end == n_layers) applies the final RMSNorm and
    the LM head and returns logits; any other stage maps hidden states to
    hidden states. The KV cache holds, per sequence and layer, the post-RoPE
    keys and the values of every processed position.
    """

    def __init__(self, cfg, weights, begin, end, dtype=np.float32):
        assert 0 <= begin <= end <= cfg.n_layers
        self.cfg, self.W, self.begin, self.end = cfg, weights, begin, end
        self.dtype = np.dtype(dtype)
        self.kv = {}   # seq_id -> {layer: (K [n, nkv, d], V [n, nkv, d])}

    # -- helpers
    def _w(self, layer, kind):
        return np.asarray(self.W(layer, kind), dtype=self.dtype)

    def _layer(self, l, x, pos, seq_id):
        """Decoder layer l on the new positions ``pos`` of one sequence."""
        cfg = self.cfg
        n = x.shape[0]
        u = rms_norm(x, self._w(l, "attn_norm"), cfg.rms_eps)
        q = (u @ self._w(l, "wq").T).reshape(n, cfg.n_heads, cfg.head_dim)
        k = (u @ self._w(l, "wk").T).reshape(n, cfg.n_kv_heads, cfg.head_dim)
        v = (u @ self._w(l, "wv").T).reshape(n, cfg.n_kv_heads, cfg.head_dim)
        cos, sin = rope_angles(pos, cfg.head_dim, cfg.rope_base)
        q = apply_rope(q, cos, sin)
        k = apply_rope(k, cos, sin)
        cache = self.kv.setdefault(seq_id, {})
        if l in cache:
            k_all = np.concatenate([cache[l][0], k], axis=0)
            v_all = np.concatenate([cache[l][1], v], axis=0)
        else:
            k_all, v_all = k, v
        cache[l] = (k_all, v_all)
        k_pos = np.arange(k_all.shape[0])
        o = attention(q, k_all, v_all, pos, k_pos)
        x = x + o @ self._w(l, "wo").T
        u = rms_norm(x, self._w(l, "ffn_norm"), cfg.rms_eps)
        x = x + swiglu(u, self._w(l, "wgate"), self._w(l, "wup"),
                       self._w(l, "wdown"))
        return x

    def _run(self, seq_id, inp, pos):
        cfg = self.cfg
        if self.begin == 0:
            x = self._w(-1, "embed")[np.asarray(inp, dtype=np.int64)]
        else:
            x = np.asarray(inp, dtype=self.dtype)
        for l in range(self.begin, self.end):
            x = self._layer(l, x, pos, seq_id)
        if self.end == cfg.n_layers:
            u = rms_norm(x, self._w(-1, "final_norm"), cfg.rms_eps)
            return u @ self._w(-1, "lm_head").T      # logits [n, V]
        return x                                    # hidden [n, H]

    def n_tokens(self, seq_id):
        c = self.kv.get(seq_id)
        if not c:
            return 0
        return next(iter(c.values()))[0].shape[0]

    # -- API mirroring the engine's calls
    def prefill(self, seq_ids, seq_lens, inp):
        """Process whole prompts. ``inp`` is packed by sequence: token ids
        [T] for the first stage, hidden [T, H] otherwise. Returns hidden
        [T, H] or logits for every position [T, V] (last stage)."""
        outs, off = [], 0
        for sid, n in zip(seq_ids, seq_lens):
            assert sid not in self.kv or self.n_tokens(sid) == 0
            outs.append(self._run(sid, inp[off:off + n], np.arange(n)))
            off += n
        return np.concatenate(outs, axis=0)

    def decode(self, seq_ids, inp):
        """One new position per sequence, reusing the cache."""
        outs = []
        for i, sid in enumerate(seq_ids):
            p = self.n_tokens(sid)
            outs.append(self._run(sid, inp[i:i + 1], np.array([p])))
        return np.concatenate(outs, axis=0)

    def drop(self, seq_id):
        self.kv.pop(seq_id, None)


def full_forward(cfg, weights, token_ids, dtype=np.float32):
    """Logits of every position of one sequence, whole model, no cache."""
    st = Stage(cfg, weights, 0, cfg.n_layers, dtype)
    return st.prefill([0], [len(token_ids)], np.asarray(token_ids))


def greedy_generate(cfg, weights, prompt, n_steps, stages=None,
                    dtype=np.float32):
    """Prefill then ``n_steps`` greedy decode steps through a pipeline of
    stages (default: one stage holding every layer).

    Returns (tokens [n_steps + 1], logits [n_steps + 1, V]): the token
    produced by prefill followed by one token per decode step."""
    if stages is None:
        stages = [(0, cfg.n_layers)]
    sts = [Stage(cfg, weights, b, e, dtype) for b, e in stages]
    x = np.asarray(prompt)
    for st in sts:
        x = st.prefill([0], [len(prompt)], x)
    logits = [x[-1]]
    toks = [int(argmax_lowest(x[-1]))]
    for _ in range(n_steps):
        x = np.array([toks[-1]], dtype=np.int32)
        for st in sts:
            x = st.decode([0], x)
        logits.append(x[0])
        toks.append(int(argmax_lowest(x[0])))
    return np.array(toks, dtype=np.int32), np.stack(logits)


# ------------------------------------------------------- size accounting

def param_count(cfg, layer_begin=0, layer_end=None, embed=None, head=None):
    """Parameters of layers [begin, end), plus the embedding (first stage)
    and the final norm + LM head (last stage) unless overridden."""
    if layer_end is None:
        layer_end = cfg.n_layers
    if embed is None:
        embed = layer_begin == 0
    if head is None:
        head = layer_end == cfg.n_layers
    h, f = cfg.hidden, cfg.ffn
    per_layer = (h * cfg.q_dim + 2 * h * cfg.kv_dim + cfg.q_dim * h
                 + 3 * h * f + 2 * h)
    n = (layer_end - layer_begin) * per_layer
    if embed:
        n += cfg.vocab * h
    if head:
        n += h + cfg.vocab * h
    return n


def image_bytes_16bit(cfg, layer_begin=0, layer_end=None):
    """Bytes of a stage's weights stored in a 16-bit format."""
    return 2 * param_count(cfg, layer_begin, layer_end)


def boundary_bytes_per_token(cfg):
    """Bytes passed between stages per token: one 16-bit hidden vector."""
    return 2 * cfg.hidden
