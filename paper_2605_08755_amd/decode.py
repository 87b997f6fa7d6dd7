"""One batch-1 decode step of a Qwen3-shaped decoder on the library's kernels.

Each layer: residual add + RMSNorm, the fused q|k|v linear (the norm inside
it when the linear offers laq.add_rmsnorm_linear), per-head q/k
RMSNorm + rotary embedding + KV-cache append, attention over the cache, the
o linear, residual add + RMSNorm, the fused gate|up linear, SiLU-and-multiply,
the down linear (whose output the next layer's first norm adds to the
residual).  The step ends with the final norm and, when one is given, the
LM head (one more caller-supplied linear, hidden -> vocabulary logits).
Argument marshalling only: every operation is a call of liblaq.so, except the
linears, which the caller supplies (the library's quantized linear, or any
other implementation of y = x W^T to compare against).
"""
import numpy as np

from . import laq

HEAD_DIM = laq.HEAD_DIM

# Qwen3-4B decoder shape (hidden, query heads, key/value heads, MLP width).
QWEN3_4B = {"layers": 36, "hidden": 2560, "heads": 32, "kv_heads": 8, "mlp": 9728,
            "eps": 1e-6, "rope_theta": 1e6, "vocab": 151936}


def rope_table(S_max, theta, device, d=HEAD_DIM):
    """fp32 [S_max][d]: cos of the d/2 rotation angles pos * theta^(-2i/d) of
    each position, then their sin (angles and cos/sin in float64)."""
    import torch
    a = np.arange(S_max, dtype=np.float64)[:, None] * theta ** (-2.0 * np.arange(d // 2) / d)[None, :]
    t = np.concatenate([np.cos(a), np.sin(a)], axis=1).astype(np.float32)
    return torch.from_numpy(t).to(device)


class DecodeStep:
    """Buffers and call sequence of one decode step.

    linears[l] = (qkv, o, gate_up, down): callables f(x, out) writing
    out = x W^T (fp16 [1][N]) for the layer's weights; a gate_up callable
    with the attribute swiglu = True writes silu(gate) * up (fp16 [1][I])
    itself (laq.linear_swiglu), and the step skips silu_mul.  norms[l] =
    (input_norm, post_attention_norm, q_norm, k_norm) fp16 vectors;
    final_norm fp16 [hidden].  k_caches / v_caches: fp16 [kv_heads][S_max][128]
    per layer (positions below the decoded one already filled).  lm_head:
    optional callable f(x, out) writing the logits out = x W^T (fp16
    [1][vocab], vocab = shape["vocab"]) from the final norm's output.
    fused_attention: the per-head q/k norm, rotary embedding, cache append
    and attention as laq.decode_attention_qkv (two kernels); False: the
    separate laq.qk_norm_rope and laq.decode_attention calls (three).

    A qkv, gate_up or lm_head callable with an attribute norm_linear =
    g(residual, delta, norm_weight, eps, residual_out, out) computes the norm
    before it itself (laq.add_rmsnorm_linear: residual_out = residual + delta,
    out = RMSNorm(residual_out) * norm_weight, then the linear, one kernel);
    the step then skips that add_rmsnorm call and continues with the residual
    in residual_out; when there is no delta the residual does not change and
    the step passes residual_out None.  The step keeps two residual buffers for this
    besides x0, which it reads in place and never writes (the first update
    goes to a buffer); `residual` is the tensor holding the current residual
    stream.  A gate_up
    callable with an attribute norm_mlp (same arguments as norm_linear, out
    receiving the down projection's output, fp16 [1][hidden]) is the whole MLP
    block after the attention: norm, gate|up, SiLU-and-multiply and down
    (laq.add_rmsnorm_mlp, one kernel); the step then skips the down call.
    An o or down callable with an attribute residual_linear = g(x,
    residual_in, residual_out, out) adds its output to the residual stream
    itself (laq.linear_residual: residual_out = residual_in + y); the next
    norm then runs with no delta, so g need not write y to out (the step
    reads only the residual; laq.linear_residual with write_out=False).
    """

    def __init__(self, shape, linears, norms, final_norm, k_caches, v_caches, device, lm_head=None,
                 fused_attention=True):
        import torch
        self.s = shape
        self.linears, self.norms, self.final_norm = linears, norms, final_norm
        self.k_caches, self.v_caches = k_caches, v_caches
        D, Hq, Hkv, I = shape["hidden"], shape["heads"], shape["kv_heads"], shape["mlp"]
        S_max = k_caches[0].shape[1]
        self.S_max = S_max
        self.cos_sin = rope_table(S_max, shape["rope_theta"], device)
        f16 = dict(dtype=torch.float16, device=device)
        self._res = [torch.zeros((1, D), dtype=torch.float32, device=device) for _ in range(2)]
        self.x0 = torch.zeros((1, D), dtype=torch.float32, device=device)  # the token's embedding
        self._r = self.x0  # the tensor holding the residual stream (x0 until the first update)
        self.h = torch.empty((1, D), **f16)
        self.qkv = torch.empty((1, (Hq + 2 * Hkv) * HEAD_DIM), **f16)
        self.q = torch.empty((Hq, HEAD_DIM), **f16)
        self.attn = torch.empty((Hq, HEAD_DIM), **f16)
        self.o = torch.empty((1, D), **f16)
        self.gu = torch.empty((1, 2 * I), **f16)
        self.m = torch.empty((1, I), **f16)
        self.down = torch.empty((1, D), **f16)
        self.out = torch.empty((1, D), **f16)
        self.lm_head = lm_head
        self.logits = torch.empty((1, shape["vocab"]), **f16) if lm_head is not None else None
        self.fused_attention = fused_attention
        nbytes = (laq.attention_qkv_workspace_bytes(Hq, Hkv, S_max) if fused_attention
                  else laq.attention_workspace_bytes(Hq, S_max))
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)

    @property
    def residual(self):
        """fp32 [1][hidden]: the residual stream as of the last call issued."""
        return self._r

    def _next(self):
        """The residual buffer the next update writes: never x0 (read-only
        input of every step) and never the current residual."""
        return self._res[1] if self._r is self._res[0] else self._res[0]

    def _in_place(self):
        """The current residual, made writable for an in-place update."""
        if self._r is self.x0:
            nxt = self._next()
            nxt.copy_(self.x0)
            self._r = nxt
        return self._r

    def _norm(self, f, delta, weight, out):
        """Residual add + RMSNorm, then f: fused into f when it offers it.
        With no delta the residual stays where it is (no residual_out)."""
        g = getattr(f, "norm_linear", None)
        if g is not None:
            if delta is None:
                g(self._r, None, weight, self.s["eps"], None, out)
                return
            nxt = self._next()
            g(self._r, delta, weight, self.s["eps"], nxt, out)
            self._r = nxt
            return
        laq.add_rmsnorm(self._in_place(), delta, weight, self.s["eps"], out=self.h)  # (writes the residual)
        f(self.h, out)

    def _linear(self, f, x, out):
        """f(x, out); returns the delta the next norm adds: out, or None when
        f added it to the residual stream itself."""
        g = getattr(f, "residual_linear", None)
        if g is None:
            f(x, out)
            return out
        nxt = self._next()
        g(x, self._r, nxt, out)
        self._r = nxt
        return None

    def run(self, pos):
        """Decode the token at position pos (attends to positions 0..pos).
        Returns the logits when the step has an LM head, else the final
        norm's output."""
        s = self.s
        Hq, Hkv, eps = s["heads"], s["kv_heads"], s["eps"]
        self._r = self.x0  # read in place: the first update writes another buffer
        delta = None
        for l, (f_qkv, f_o, f_gu, f_down) in enumerate(self.linears):
            w_in, w_post, qn, kn = self.norms[l]
            self._norm(f_qkv, delta, w_in, self.qkv)
            if self.fused_attention:
                laq.decode_attention_qkv(self.qkv, qn, kn, self.cos_sin, pos, Hq, Hkv, eps, self.k_caches[l],
                                         self.v_caches[l], out=self.attn, workspace=self.workspace)
            else:
                laq.qk_norm_rope(self.qkv, qn, kn, self.cos_sin, pos, Hq, Hkv, eps, self.k_caches[l],
                                 self.v_caches[l], q_out=self.q)
                laq.decode_attention(self.q, self.k_caches[l], self.v_caches[l], pos + 1, out=self.attn,
                                     workspace=self.workspace)
            delta = self._linear(f_o, self.attn.view(1, Hq * HEAD_DIM), self.o)
            mlp = getattr(f_gu, "norm_mlp", None)
            if mlp is not None:
                nxt = self._next()
                mlp(self._r, delta, w_post, eps, nxt, self.down)
                self._r = nxt
                delta = self.down
                continue
            if getattr(f_gu, "swiglu", False):
                self._norm(f_gu, delta, w_post, self.m)
            else:
                self._norm(f_gu, delta, w_post, self.gu)
                laq.silu_mul(self.gu, out=self.m)
            delta = self._linear(f_down, self.m, self.down)
        if self.lm_head is not None and getattr(self.lm_head, "norm_linear", None) is not None:
            self._norm(self.lm_head, delta, self.final_norm, self.logits)
            return self.logits
        laq.add_rmsnorm(self._in_place(), delta, self.final_norm, eps, out=self.out)
        if self.lm_head is None:
            return self.out
        self.lm_head(self.out, self.logits)
        return self.logits
