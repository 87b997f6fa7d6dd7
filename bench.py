"""Decode-step W3G128 linear stack on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

A step is one decode step's worth of quantized linears: the 36-layer
Qwen3-4B-shaped stack (q, k, v, o, gate, up, down per layer) at M = 1,
captured once into a HIP graph and replayed.  Projections that read the same
activation run as one call on row-concatenated weights (q|k|v and gate|up),
so a layer is 4 dependent calls of laq_linear_w3g128 (144 per step); the
one-call-per-projection figure (252 per step) is reported beside it.
Weights are synthetic (seeded N(0, 0.02) with 1% x10 outliers, drawn on the
GPU) and quantized by laq_quantize_w3g128 before timing; activations are
seeded N(0, 1); everything is resident in HBM before the timed region.

Prints one JSON line.  `value` is the effective weight-stream bandwidth of
the whole step (packed codes + scales + zeros bytes / step time, graph wall
time); `roofline` compares the linear kernel's own duration (HIP events at
kernel start/end) with the 8 TB/s HBM peak; `cpu_baseline` times the CPU
oracle on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs/decode-step linear stack + effective weight GB/s (% of HBM peak), M=1"
HBM_PEAK_GBS = 8000.0
GROUP = 128


KERNEL_SOURCES = ("paper_2605_08755_amd/csrc/linear.hip", "paper_2605_08755_amd/csrc/laq_internal.h")


def kernel_code_digest():
    """sha256 of the GEMV's sources with comments and blank space removed, so
    that a comment-only edit keeps the HBM-counter record valid while any
    change of the code invalidates it."""
    import hashlib
    import re
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per GEMV launch from the committed rocprofv3 counter runs
    (profiles/hbm_traffic.json), or None when the kernel code has changed
    since those counters were taken."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
        digest = kernel_code_digest()
    except (OSError, KeyError, ValueError):
        return None
    if digest != rec.get("kernel_code_digest"):
        return None
    return rec


def bytes_per_weight(bits):
    # codes + fp16 scale + uint8 zero per 128-group
    return bits / 8 + 2 / GROUP + 1 / GROUP


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# Projections that read the same activation are fused into one call by
# concatenating their weights along N (quantization is per row, so the
# concatenated quantization equals the separate ones): q|k|v and gate|up.
FUSED = {"qkv": ("q", "k", "v"), "gateup": ("gate", "up")}


class Stack:
    """All quantized projections of a workload, resident on the GPU.

    fused=True: one call per decode stage that shares an input (q|k|v, o,
    gate|up, down: 4 per layer); fused=False: one call per projection.
    """

    def __init__(self, workload, device, bits_list=(3,), keep_fp16=False, fused=True):
        import torch
        from paper_2605_08755_amd import inputs, laq
        spec = inputs.WORKLOADS[workload]
        self.workload = workload
        self.layers = spec["layers"]
        self.projs = spec["projs"]
        self.device = device
        self.fused = fused
        self.q = {b: [] for b in bits_list}
        self.fp16 = [] if keep_fp16 else None
        self.shapes = []
        names = [p[0] for p in self.projs]
        groups = []
        if fused and all(n in names for members in FUSED.values() for n in members):
            done = set()
            for name in names:
                if name in done:
                    continue
                for fname, members in FUSED.items():
                    if name in members:
                        groups.append((fname, members))
                        done.update(members)
                        break
                else:
                    groups.append((name, (name,)))
                    done.add(name)
        else:
            groups = [(n, (n,)) for n in names]
        self.groups = groups
        for layer in range(self.layers):
            for gname, members in groups:
                parts = []
                for name in members:
                    pi = names.index(name)
                    _, N, K = self.projs[pi]
                    parts.append(inputs.weights_torch(N, K, seed=layer * 16 + pi, device=device))
                w = parts[0] if len(parts) == 1 else torch.cat(parts, dim=0)
                del parts
                N, K = w.shape
                for b in bits_list:
                    self.q[b].append(laq.quantize(w, b))
                if keep_fp16:
                    self.fp16.append(w)
                del w
                self.shapes.append((layer, gname, N, K))
        torch.cuda.synchronize()
        self.x = {}
        slots = sorted({(layer, inputs.X_SLOT.get(FUSED.get(name, (name,))[0], 0), K)
                        for (layer, name, N, K) in self.shapes})
        for (layer, slot, K) in slots:
            self.x[(layer, slot)] = inputs.activations_torch(16, K, seed=layer * 8 + slot, device=device)
        self.y = [torch.empty((16, N), dtype=torch.float16, device=device) for (_, _, N, _) in self.shapes]
        self.slot_of = [inputs.X_SLOT.get(FUSED.get(name, (name,))[0], 0) for (_, name, _, _) in self.shapes]

    def weights(self):
        return sum(N * K for (_, _, N, K) in self.shapes)

    def weight_bytes(self, bits):
        return self.weights() * bytes_per_weight(bits)

    def step(self, M, bits, events=None):
        from paper_2605_08755_amd import laq
        for i, (layer, name, N, K) in enumerate(self.shapes):
            q, s, z = self.q[bits][i]
            if events is not None:
                laq.profile_next_launch(*events[i])
            laq.linear(self.x[(layer, self.slot_of[i])][:M], q, s, z, bits, out=self.y[i][:M])


def grouped_step(stack, M, bits):
    """One decode step of an unfused stack with the calls that share a stage
    issued as one grouped launch each: q,k,v | o | gate,up | down."""
    from paper_2605_08755_amd import laq
    idx = {}
    for i, (layer, name, N, K) in enumerate(stack.shapes):
        idx[(layer, name)] = i
    for layer in range(stack.layers):
        for members in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
            ii = [idx[(layer, n)] for n in members]
            calls = [(stack.x[(layer, stack.slot_of[i])][:M],) + tuple(stack.q[bits][i]) for i in ii]
            outs = [stack.y[i][:M] for i in ii]
            if len(ii) == 1:
                laq.linear(*calls[0], bits, out=outs[0])
            else:
                laq.linear_group(calls, bits, outs=outs)


def time_graph(stack, M, bits, steps, warmup, step_fn=None):
    """Capture one step into a HIP graph; time `steps` replays."""
    import torch
    if step_fn is None:
        def step_fn():
            stack.step(M, bits)
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    step_fn()  # eager warm-up (loads code objects)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        step_fn()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / steps
    del g
    return ms, wall


def replay_distribution(stack, M, bits, reps=100, warmup=10):
    """Per-replay step times of the captured step: `reps` replays, each
    bracketed by its own pair of events on the replay stream, after `warmup`
    replays; median and 10th / 90th percentiles in microseconds.  A separate
    pass from the headline's timed region (the events between replays add a
    little to each one)."""
    import torch
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    stack.step(M, bits)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        stack.step(M, bits)
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            g.replay()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record(stream)
            g.replay()
            b.record(stream)
    torch.cuda.synchronize()
    us = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
    pick = lambda f: us[min(len(us) - 1, int(round(f * (len(us) - 1))))]
    del g
    return {"reps": reps, "median_us": round(pick(0.5), 2), "p10_us": round(pick(0.1), 2),
            "p90_us": round(pick(0.9), 2), "min_us": round(us[0], 2), "max_us": round(us[-1], 2)}


def time_calls_graph(fn, reps=5):
    """Capture the launches fn() makes into a HIP graph and time `reps`
    replays on the current stream: ms per pass, with no host launch gaps."""
    import torch
    fn()  # eager warm-up
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        fn()
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del g
    return ms


def time_fp16_graph(stack, M, steps, warmup):
    """The same step with the fp16 weights through torch's dense GEMM
    (hipBLASLt): the unquantized reference for the quantized speed-up."""
    import torch

    def step():
        for i, (layer, name, N, K) in enumerate(stack.shapes):
            torch.mm(stack.x[(layer, stack.slot_of[i])][:M], stack.fp16[i].t(), out=stack.y[i][:M])

    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    step()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        step()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del g
    return ms


def decode_step_extra(stack, dev, steps, context=1024):
    """One batch-1 decode step of the Qwen3-4B-shaped decoder (36 layers:
    norms, rotary embedding, attention over a synthetic KV cache of `context`
    positions, SiLU-and-multiply, the stack's linears, the final norm and the
    LM head over Qwen3-4B's 151936-token vocabulary), the token at position
    context - 1, captured in a HIP graph.  Variants: W3 linears and a W3 LM
    head; W3 with the gate|up + SiLU linear and a W3 or an fp16 LM head; the
    same with the norms before q|k|v and gate|up inside those linears
    (laq.add_rmsnorm_linear), also with o and down adding their outputs to
    the residual stream (laq.linear_residual) and with the MLP block in one
    launch (laq.add_rmsnorm_mlp); fp16 weights everywhere through torch's dense
    GEMM (the unquantized reference).  The paper does not say whether its decoding benchmark
    quantizes the LM head, hence both heads.  Attention is the fused
    q/k-norm + rotary + attention call except in the _separate_attention
    variant (qk-norm-rope, attention partials, combine: three kernels)."""
    import torch
    from paper_2605_08755_amd import decode, inputs, laq
    shape = dict(decode.QWEN3_4B)
    assert stack.workload == "stack4b" and len(stack.shapes) == 4 * shape["layers"]
    g = torch.Generator(device=dev)
    g.manual_seed(inputs.ENTROPY * 1000 + 900000)

    def vec(n):
        return (1.0 + 0.1 * torch.randn((n,), generator=g, device=dev)).to(torch.float16)

    D, Hkv, V = shape["hidden"], shape["kv_heads"], shape["vocab"]
    norms = [(vec(D), vec(D), vec(128), vec(128)) for _ in range(shape["layers"])]
    caches = [torch.randn((2, Hkv, context, 128), generator=g, device=dev).to(torch.float16)
              for _ in range(shape["layers"])]
    w_head = inputs.weights_torch(V, D, seed=999999, device=dev)
    q_head = laq.quantize(w_head, 3)

    def w3_lin(i):
        q, sc, z = stack.q[3][i]
        return lambda x, out: laq.linear(x, q, sc, z, 3, out=out)

    def fp16_lin(i):
        w = stack.fp16[i]
        return lambda x, out: torch.mm(x, w.t(), out=out)

    I = shape["mlp"]
    swiglu_w = {}

    def w3_swiglu_lin(i):
        # gate|up rows interleaved (gate j, up j), quantized per row as before
        if i % 4 != 2:
            return w3_lin(i)
        w = stack.fp16[i]
        q, sc, z = swiglu_w[i] = laq.quantize(torch.stack([w[:I], w[I:]], dim=1).reshape(2 * I, -1).contiguous(), 3)
        f = lambda x, out: laq.linear_swiglu(x, q, sc, z, 3, out=out)
        f.swiglu = True
        return f

    def with_norm(f, q, sc, z, swiglu=False):
        # the norm before this linear computed inside it (laq.add_rmsnorm_linear)
        f.norm_linear = lambda res, delta, w, eps, res_out, out: laq.add_rmsnorm_linear(
            res, delta, w, eps, q, sc, z, 3, swiglu=swiglu, out=out, residual_out=res_out)
        return f

    def w3_norm_lin(i):
        if i % 4 == 2:
            f = w3_swiglu_lin(i)
            return with_norm(f, *swiglu_w[i], swiglu=True)
        f = w3_lin(i)
        return with_norm(f, *stack.q[3][i]) if i % 4 == 0 else f

    def w3_residual_lin(i):
        # as w3_norm_lin, with o and down adding their outputs to the residual
        # stream themselves (laq.linear_residual), so the norms take no delta
        f = w3_norm_lin(i)
        if i % 4 in (1, 3):
            q, sc, z = stack.q[3][i]
            f.residual_linear = lambda x, r_in, r_out, out: laq.linear_residual(x, q, sc, z, r_in, r_out, 3,
                                                                                write_out=False)
        return f

    mlp_ws = laq.mlp_workspace(D, I, dev)  # stream-ordered calls share it

    def w3_merged_mlp_lin(i):
        # as w3_norm_lin, with norm + gate|up + SiLU + down of the MLP block in
        # one launch (laq.add_rmsnorm_mlp; the down callable is then unused)
        f = w3_norm_lin(i)
        if i % 4 == 2:
            gu, dn = swiglu_w[i], stack.q[3][i + 1]
            f.norm_mlp = lambda res, delta, w, eps, res_out, out: laq.add_rmsnorm_mlp(
                res, delta, w, eps, gu, dn, mlp_ws, out=out, residual_out=res_out)
        return f

    # (the final norm stays a separate call: inside the 151936-row head the
    # prologue cost more than the norm's own launch with 256-thread blocks,
    # and the same, 987-991 us per token either way, with 512-thread ones)
    head_w3 = lambda x, out: laq.linear(x, *q_head, 3, out=out)
    head_fp16 = lambda x, out: torch.mm(x, w_head.t(), out=out)
    out = {"context": context, "layers": shape["layers"], "vocab": V}
    variants = (("w3", w3_lin, head_w3, True), ("w3_fused_swiglu", w3_swiglu_lin, head_w3, True),
                ("w3_fused_swiglu_fused_norms", w3_norm_lin, head_w3, True),
                ("w3_fused_norms_residual", w3_residual_lin, head_w3, True),
                ("w3_merged_mlp", w3_merged_mlp_lin, head_w3, True),
                ("w3_fused_swiglu_separate_attention", w3_swiglu_lin, head_w3, False),
                ("w3_fused_swiglu_fp16_head", w3_swiglu_lin, head_fp16, True), ("fp16", fp16_lin, head_fp16, True))
    for name, mk, head, fused_attention in variants:
        lins = [tuple(mk(4 * l + j) for j in range(4)) for l in range(shape["layers"])]
        step = decode.DecodeStep(shape, lins, norms, vec(D), [c[0] for c in caches], [c[1] for c in caches], dev,
                                 lm_head=head, fused_attention=fused_attention)
        step.x0.copy_(torch.randn((1, D), generator=g, device=dev))
        ms, _ = time_graph(stack, 1, 3, steps, 5, step_fn=lambda: step.run(context - 1))
        out[name] = {"us": round(ms * 1e3, 1), "tokens_per_s": round(1e3 / ms, 1)}
        del step
    swiglu_w.clear()
    for name in ("w3", "w3_fused_swiglu", "w3_fused_swiglu_fused_norms", "w3_fused_norms_residual", "w3_merged_mlp",
                 "w3_fused_swiglu_fp16_head"):
        out[name + "_speedup_vs_fp16"] = round(out["fp16"]["us"] / out[name]["us"], 3)

    # Attention alone: a HIP graph of the 36 layers' attention calls (each
    # layer's own cache, the token at position context - 1), back to back as in
    # the step, µs per call and the cache bytes read per second.
    Hq, hd = shape["heads"], 128
    qkv = torch.randn(((Hq + 2 * Hkv) * hd,), generator=g, device=dev).to(torch.float16)
    cs = decode.rope_table(context, shape["rope_theta"], dev)
    att = torch.empty((Hq, hd), dtype=torch.float16, device=dev)
    q_sep = torch.empty((Hq, hd), dtype=torch.float16, device=dev)
    ws_f = torch.empty(laq.attention_qkv_workspace_bytes(Hq, Hkv, context), dtype=torch.uint8, device=dev)
    ws_s = torch.empty(laq.attention_workspace_bytes(Hq, context), dtype=torch.uint8, device=dev)
    pos = context - 1
    cache_bytes = 2 * Hkv * context * hd * 2

    def fused():
        for l in range(shape["layers"]):
            qn, kn = norms[l][2], norms[l][3]
            laq.decode_attention_qkv(qkv, qn, kn, cs, pos, Hq, Hkv, 1e-6, caches[l][0], caches[l][1], out=att,
                                     workspace=ws_f)

    def separate():
        for l in range(shape["layers"]):
            qn, kn = norms[l][2], norms[l][3]
            laq.qk_norm_rope(qkv, qn, kn, cs, pos, Hq, Hkv, 1e-6, caches[l][0], caches[l][1], q_out=q_sep)
            laq.decode_attention(q_sep, caches[l][0], caches[l][1], pos + 1, out=att, workspace=ws_s)

    att_out = {}
    for name, fn in (("fused", fused), ("separate", separate)):
        us = time_calls_graph(fn, reps=20) * 1e3 / shape["layers"]
        att_out[name] = {"us_per_layer": round(us, 3), "cache_TBps": round(cache_bytes / (us * 1e-6) / 1e12, 3)}
    out["attention_graph"] = att_out

    # The MLP block alone: a HIP graph of the 36 layers' MLP blocks (each
    # layer's own weights), as two launches (norm + gate|up + SiLU, then down)
    # and as one (laq.add_rmsnorm_mlp), µs per layer.
    res = [torch.randn((1, D), generator=g, device=dev) for _ in range(2)]
    o = torch.randn((1, D), generator=g, device=dev).to(torch.float16)
    m = torch.empty((1, I), dtype=torch.float16, device=dev)
    y = torch.empty((1, D), dtype=torch.float16, device=dev)
    gu_w = []
    for l in range(shape["layers"]):
        w = stack.fp16[4 * l + 2]
        gu_w.append(laq.quantize(torch.stack([w[:I], w[I:]], dim=1).reshape(2 * I, -1).contiguous(), 3))

    def two_launch():
        for l in range(shape["layers"]):
            laq.add_rmsnorm_linear(res[0], o, norms[l][1], 1e-6, *gu_w[l], 3, swiglu=True, out=m,
                                   residual_out=res[1])
            laq.linear(m, *stack.q[3][4 * l + 3], 3, out=y)

    def one_launch():
        for l in range(shape["layers"]):
            laq.add_rmsnorm_mlp(res[0], o, norms[l][1], 1e-6, gu_w[l], stack.q[3][4 * l + 3], mlp_ws, out=y,
                                residual_out=res[1])

    out["mlp_graph"] = {name: {"us_per_layer": round(time_calls_graph(fn, reps=20) * 1e3 / shape["layers"], 3)}
                        for name, fn in (("two_launch", two_launch), ("merged", one_launch))}
    return out


def stack32b_extra(dev, steps):
    """The 64-layer Qwen3-32B-shaped stack: W3 decode-step time at M = 1 and
    16, and quantize throughput over all of its fp16 weights."""
    import torch
    from paper_2605_08755_amd import laq
    t0 = time.perf_counter()
    st = Stack("stack32b", dev, bits_list=(3,), keep_fp16=True, fused=True)
    log("stack32b built in %.1f s: %d calls per step, %.2f G weights"
        % (time.perf_counter() - t0, len(st.shapes), st.weights() / 1e9))
    wb = st.weight_bytes(3)
    out = {"layers": st.layers, "weights_per_step": st.weights(), "weight_bytes_per_step": int(round(wb)),
           "linears_per_step": len(st.shapes)}
    for M in (1, 16):
        ms, _ = time_graph(st, M, 3, steps, 5)
        gbs = wb / (ms * 1e-3) / 1e9
        out["w3_m%d" % M] = {"us": round(ms * 1e3, 1), "GBps": round(gbs, 1),
                             "pct_of_hbm_peak": round(gbs / HBM_PEAK_GBS * 100, 2)}
    def quantize_all():
        for i, w in enumerate(st.fp16):
            laq.quantize(w, 3, out=st.q[3][i])
    qms = time_calls_graph(quantize_all, reps=3)
    out["quantize_w3"] = {"ms": round(qms, 3),
                          "GBps": round(st.weights() * (2 + bytes_per_weight(3)) / (qms * 1e-3) / 1e9, 1)}
    log("stack32b:", out)
    del st
    torch.cuda.empty_cache()
    return out


def per_call_graph(stack, M, bits, reps=20):
    """Per call shape: a HIP graph of that shape's calls of every layer, back
    to back (distinct weights, as in the step); µs per call and algorithmic
    GB/s.  The one per-projection figure that includes no event or launch
    overhead beyond the dependent-launch gap of the step itself."""
    import torch
    from paper_2605_08755_amd import laq
    out = {}
    for gname in [g[0] for g in stack.groups]:
        idx = [i for i, sh in enumerate(stack.shapes) if sh[1] == gname]
        N, K = stack.shapes[idx[0]][2], stack.shapes[idx[0]][3]

        def fn():
            for i in idx:
                layer = stack.shapes[i][0]
                q, sc, z = stack.q[bits][i]
                laq.linear(stack.x[(layer, stack.slot_of[i])][:M], q, sc, z, bits, out=stack.y[i][:M])
        ms = time_calls_graph(fn, reps=reps)
        us = ms * 1e3 / len(idx)
        out[gname] = {"N": N, "K": K, "us": round(us, 3),
                      "GBps": round(N * K * bytes_per_weight(bits) / (us * 1e-6) / 1e9, 1)}
    return out


def single_extra(dev, reps=20):
    """The single 1024 x 1024 W3G128 linear at M = 1: µs per call with the
    same weights every call (0.42 MB, cache-resident: the latency-bound
    figure), and over 2400 rotated copies (1.0 GB streamed from HBM per pass)
    for an HBM rate; quantize µs per call."""
    import torch
    from paper_2605_08755_amd import inputs, laq
    N = K = 1024
    w = inputs.weights_torch(N, K, seed=77, device=dev)
    q, sc, z = laq.quantize(w, 3)
    x = inputs.activations_torch(1, K, seed=77, device=dev)
    y = torch.empty((1, N), dtype=torch.float16, device=dev)

    def same():
        for _ in range(1000):
            laq.linear(x, q, sc, z, 3, out=y)
    us_same = time_calls_graph(same, reps=reps) * 1e3 / 1000
    copies = 2400
    ws = [laq.quantize(inputs.weights_torch(N, K, seed=1000 + i, device=dev), 3) for i in range(copies)]

    def rotated():
        for (qq, ss, zz) in ws:
            laq.linear(x, qq, ss, zz, 3, out=y)
    us_rot = time_calls_graph(rotated, reps=3) * 1e3 / copies
    qout = (torch.empty_like(q), torch.empty_like(sc), torch.empty_like(z))

    def quant():
        for _ in range(200):
            laq.quantize(w, 3, out=qout)
    us_q = time_calls_graph(quant, reps=reps) * 1e3 / 200
    del ws
    torch.cuda.empty_cache()
    wb = N * K * bytes_per_weight(3)
    return {"shape": "N=1024, K=1024, M=1, W3G128", "weight_bytes": int(wb),
            "linear_us_same_weights": round(us_same, 3),
            "linear_us_rotated_1GB": round(us_rot, 3),
            "linear_GBps_rotated": round(wb / (us_rot * 1e-6) / 1e9, 1),
            "quantize_us": round(us_q, 3)}


def trace_run(args, dev):
    """Workload for rocprofv3 --kernel-trace: the headline step (W3, M = 1,
    144 dependent GEMV launches), one eager warm-up step, then --warmup +
    --steps replays of its HIP graph, nothing else.  --summarize-trace reads
    the resulting kernel_trace.csv."""
    import torch
    stack = Stack(args.workload, dev, bits_list=(3,), fused=not args.unfused)
    ms, _ = time_graph(stack, 1, 3, args.steps, args.warmup)
    print("trace run: %d launches per step, %d graph replays (%d warm-up), %.2f us/step by HIP events"
          % (len(stack.shapes), args.steps + args.warmup, args.warmup, ms * 1e3), flush=True)


def summarize_trace(path, launches, steps):
    """Markdown summary of a rocprofv3 kernel_trace.csv from --trace-run:
    per-dispatch durations of the GEMV over the last `steps` graph replays
    (by call shape: grid size), and per replay the span from the first
    dispatch's start to the last one's end."""
    import csv
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if "linear" in r["Kernel_Name"]:
                rows.append(r)
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    rows = rows[-launches * steps:]
    assert len(rows) == launches * steps, (len(rows), launches * steps)
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    spans, sums, gaps = [], [], []
    for i in range(steps):
        st = rows[i * launches:(i + 1) * launches]
        spans.append((int(st[-1]["End_Timestamp"]) - int(st[0]["Start_Timestamp"])) / 1e3)
        sums.append(sum(durs[i * launches:(i + 1) * launches]))
    by = {}
    for r, d in zip(rows, durs):
        name = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("void ", "")
        key = (name.split("(")[0][-60:], r.get("Grid_Size_X", r.get("Grid_Size", "")))
        by.setdefault(key, []).append(d)
    med = lambda v: sorted(v)[len(v) // 2]
    lines = ["| kernel (name tail) | grid | dispatches | avg µs | p50 µs | min µs |", "|---|---|---|---|---|---|"]
    for (k, g), v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        lines.append("| %s | %s | %d | %.3f | %.3f | %.3f |" % (k, g, len(v), sum(v) / len(v), med(v), min(v)))
    lines.append("")
    lines.append("Per graph replay (%d replays, %d GEMV dispatches each): first start to last end %.1f µs "
                 "(p50 %.1f), i.e. %.3f µs per launch; sum of dispatch durations %.1f µs (p50 %.1f), "
                 "%.3f µs per dispatch."
                 % (steps, launches, sum(spans) / steps, med(spans), sum(spans) / steps / launches,
                    sum(sums) / steps, med(sums), sum(sums) / steps / launches))
    return "\n".join(lines)


def kernel_table(path):
    """Markdown table of every library kernel in a rocprofv3 kernel_trace.csv
    (any run of this file): per kernel name and grid, dispatches, average,
    median and minimum End - Start in µs, and the total in ms."""
    import csv
    by = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"]
            if "laq::" not in name:
                continue
            name = name.replace("(anonymous namespace)::", "").replace("void ", "").replace("laq::", "")
            key = (name.split("(")[0], r.get("Grid_Size_X", r.get("Grid_Size", "")),
                   r.get("Workgroup_Size_X", r.get("Workgroup_Size", "")))
            by.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    med = lambda v: sorted(v)[len(v) // 2]
    lines = ["| kernel | grid | block | dispatches | avg µs | p50 µs | min µs | total ms |",
             "|---|---|---|---|---|---|---|---|"]
    for (k, g, b), v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        lines.append("| %s | %s | %s | %d | %.3f | %.3f | %.3f | %.2f |"
                     % (k, g, b, len(v), sum(v) / len(v), med(v), min(v), sum(v) / 1e3))
    return "\n".join(lines)


def pmc_summary(fetch_csv, write_csv, launches, steps):
    """Per-launch HBM bytes of the GEMV from two rocprofv3 --pmc runs of
    --profile-run (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each
    scaled by what the counter reads for the 256 MiB device copy that
    --profile-run performs first.  Also per library kernel and grid: the
    dispatches and the mean raw counter values (KiB, unscaled)."""
    import csv

    def load(path, counter, per):
        copy, lin = [], []
        with open(path) as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name", counter) != counter:
                    continue
                v = float(r["Counter_Value"])
                name = r["Kernel_Name"]
                if "laq::" in name:
                    tail = name.replace("(anonymous namespace)::", "").replace("void ", "").replace("laq::", "")
                    per.setdefault((tail.split("(")[0], r.get("Grid_Size", "")), {}).setdefault(counter, []).append(v)
                if "linear" in name:
                    lin.append(v)
                elif "copy" in name.lower() or "elementwise" in name.lower():
                    copy.append(v)
        return copy, lin
    per = {}
    cf, lf = load(fetch_csv, "FETCH_SIZE", per)
    cw, lw = load(write_csv, "WRITE_SIZE", per)
    nbytes_kib = (256 << 20) / 1024
    fscale = nbytes_kib / max(cf)
    wscale = nbytes_kib / max(cw)
    lf, lw = lf[-launches * steps:], lw[-launches * steps:]
    fetch = sum(lf) / len(lf) * fscale * 1024
    write = sum(lw) / len(lw) * wscale * 1024
    return {"fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
            "calibration": "256 MiB device copy: FETCH_SIZE %.0f KiB, WRITE_SIZE %.0f KiB (read and written: "
                           "%.0f KiB each)" % (max(cf), max(cw), nbytes_kib),
            "fetch_bytes_per_launch": int(round(fetch)), "write_bytes_per_launch": int(round(write)),
            "hbm_bytes_per_launch": int(round(fetch + write)), "dispatches": len(lf),
            "per_kernel_raw_kib": [{"kernel": k, "grid": g,
                                    "dispatches": len(c.get("FETCH_SIZE", [])),
                                    "FETCH_SIZE": round(sum(c["FETCH_SIZE"]) / len(c["FETCH_SIZE"]), 1)
                                    if c.get("FETCH_SIZE") else None,
                                    "WRITE_SIZE": round(sum(c["WRITE_SIZE"]) / len(c["WRITE_SIZE"]), 1)
                                    if c.get("WRITE_SIZE") else None}
                                   for (k, g), c in sorted(per.items())]}


def kernel_durations(stack, M, bits, reps):
    """Per-launch kernel durations (ms) from events recorded at kernel start/end."""
    import torch
    n = len(stack.shapes)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in ev:  # materialize the underlying hipEvents
        a.record()
        b.record()
    torch.cuda.synchronize()
    tot = [0.0] * n
    for _ in range(reps):
        stack.step(M, bits, events=ev)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            tot[i] += a.elapsed_time(b)
    return [t / reps for t in tot]


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_layer_rate(budget_s, projs=None):
    """(GB/s, seconds per layer, repetitions, weights) of the oracle's fp64
    linear over layer 0 of the Qwen3-4B stack (or the projections named)."""
    import oracle
    from paper_2605_08755_amd import inputs
    cases = []
    for pi, (name, N, K) in enumerate(inputs.QWEN3_4B):
        if projs is not None and name not in projs:
            continue
        w = inputs.weights(N, K, cfg=3, layer=0, proj=pi)
        codes, s, z = oracle.quantize(w, 3)
        x = inputs.activations(1, K, cfg=3, layer=0, slot=inputs.X_SLOT[name])
        cases.append((x, codes, s, z, N * K))
        del w
    weights = sum(c[4] for c in cases)
    reps = 0
    t0 = time.perf_counter()
    while True:
        for (x, codes, s, z, _) in cases:
            oracle.linear(x, codes, s, z)
        reps += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = (time.perf_counter() - t0) / reps
    return weights * bytes_per_weight(3) / dt / 1e9, dt, reps, weights


def cpu_baseline(budget_s=12.0):
    """The CPU oracle (as it stands) on a bounded sample: layer 0 of the
    Qwen3-4B stack (7 projections, M = 1), repeated for ~budget_s seconds on
    all host threads; and the k projection alone on one thread (a child
    process with OMP_NUM_THREADS=1)."""
    import subprocess
    import oracle
    gbs, dt, reps, weights = _oracle_layer_rate(budget_s)
    one = None
    try:
        code = ("import sys, json; sys.path.insert(0, %r); import bench, oracle; "
                "r = bench._oracle_layer_rate(4.0, projs=('k',)); "
                "print(json.dumps([r[0], r[1], r[2], r[3], oracle.num_threads()]))" % ROOT)
        env = dict(os.environ, OMP_NUM_THREADS="1")
        r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
        v = json.loads(r.stdout.strip().splitlines()[-1])
        one = {"value": round(v[0], 4), "unit": "GB/s", "cores": v[4],
               "sample": "the k projection of layer 0 (1024 x 2560, %d weights), %d repetitions, %.1f ms each"
                         % (v[3], v[2], v[1] * 1e3)}
    except Exception as e:  # the one-thread figure is informative only
        one = {"error": str(e)[:200]}
    return {"value": round(gbs, 3), "unit": "GB/s", "cores": oracle.num_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": "layer 0 of the 36-layer Qwen3-4B-shaped stack: 7 W3G128 projections "
                      "(%d weights) at M=1, oracle fp64 linear on its own codes, %d repetitions "
                      "in %.1f s; %.1f ms per layer, i.e. %.0f ms per 36-layer step"
                      % (weights, reps, dt * reps, dt * 1e3, dt * 36e3),
            "us_per_step_equiv": round(dt * 36e6, 1),
            "one_thread": one}


def profile_run(args, dev):
    """Workload for counter collection: a plain device copy of known size
    (its FETCH_SIZE / WRITE_SIZE calibrate the counters) followed by eager
    steps of the W3 stack at M = --profile-m activation rows (one dispatch
    per linear call)."""
    import torch
    nbytes = 256 << 20
    a = torch.empty(nbytes // 2, dtype=torch.float16, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    del a, b
    stack = Stack(args.workload, dev, bits_list=(3,), fused=not args.unfused)
    for _ in range(args.steps):
        stack.step(args.profile_m, 3)
    torch.cuda.synchronize()
    print("profile run: copy 3 x %d bytes; %d steps x %d linear calls at M=%d; %d weight bytes per step"
          % (nbytes, args.steps, len(stack.shapes), args.profile_m, int(stack.weight_bytes(3))), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="stack4b")
    ap.add_argument("--profile-reps", type=int, default=5)
    ap.add_argument("--no-sweep", action="store_true", help="skip the M x bits sweep and quantize timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-run", action="store_true",
                    help="for rocprofv3: a 256 MiB device copy (counter calibration) and --steps eager "
                         "W3 M=1 stack steps; prints a short summary instead of the JSON line")
    ap.add_argument("--profile-m", type=int, default=1, help="activation rows of the --profile-run steps (1..16)")
    ap.add_argument("--unfused", action="store_true",
                    help="one call per projection (7 per layer) instead of one per shared-input stage (4)")
    ap.add_argument("--trace-run", action="store_true",
                    help="for rocprofv3 --kernel-trace: the headline step's graph, --warmup + --steps replays only")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print a markdown summary of a --trace-run kernel trace (last --steps replays) and exit")
    ap.add_argument("--kernel-table", metavar="KERNEL_TRACE_CSV",
                    help="print per-kernel dispatch statistics of any kernel trace of this file and exit")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the per-launch HBM bytes of --profile-run counter collections and exit")
    ap.add_argument("--launches", type=int, default=144, help="GEMV launches per step (for the summaries)")
    args = ap.parse_args()

    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.launches, args.steps))
        return
    if args.kernel_table:
        print(kernel_table(args.kernel_table))
        return
    if args.pmc_summary:
        rec = pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.launches, args.steps)
        rec["kernel_code_digest"] = kernel_code_digest()
        print(json.dumps(rec, indent=1))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this library's path runs on a single MI355X "
              "(multi-GPU sharding is a design note, not built); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_08755_amd import laq
    laq.lib()  # fails loudly when liblaq.so is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.profile_run:
        profile_run(args, dev)
        return
    if args.trace_run:
        trace_run(args, dev)
        return

    bits_list = (3,) if args.no_sweep else (3, 4)
    log("building %s (bits %s) ..." % (args.workload, bits_list))
    t0 = time.perf_counter()
    stack = Stack(args.workload, dev, bits_list=bits_list, keep_fp16=not args.no_sweep, fused=not args.unfused)
    log("built in %.1f s: %d linear calls per step, %.3f G weights" % (time.perf_counter() - t0, len(stack.shapes), stack.weights() / 1e9))

    # ---- headline: W3, M = 1, graph replay
    wbytes = stack.weight_bytes(3)
    ms, wall = time_graph(stack, 1, 3, args.steps, args.warmup)
    value = wbytes / (ms * 1e-3) / 1e9
    log("W3 M=1: %.1f us/step, %.1f GB/s (%.1f%% of 8 TB/s)" % (ms * 1e3, value, value / HBM_PEAK_GBS * 100))

    # ---- kernel-level.  The step is nothing but the GEMV's 144 dependent
    # launches, back to back in the graph, so the timed region's HIP events
    # (on the replay stream) divided by the launch count give the kernel's
    # average launch duration.  Per call shape, events recorded at each
    # kernel's own start and end (eager launches) give the breakdown.
    n_launch = len(stack.shapes)
    avg_launch_ms = ms / n_launch
    achieved = wbytes / n_launch / (avg_launch_ms * 1e-3) / 1e9
    durs = kernel_durations(stack, 1, 3, args.profile_reps)
    ksum_ms = sum(durs)
    per_proj = {}
    for (layer, name, N, K), d in zip(stack.shapes, durs):
        p = per_proj.setdefault(name, {"N": N, "K": K, "us": 0.0, "n": 0})
        p["us"] += d * 1e3
        p["n"] += 1
    for name, p in per_proj.items():
        p["us"] = round(p["us"] / p["n"], 3)
        p["GBps"] = round(p["N"] * p["K"] * bytes_per_weight(3) / (p["us"] * 1e-6) / 1e9, 1)
        del p["n"]
    log("avg launch %.3f us (graph) -> %.1f GB/s per launch; eager kernel events: sum %.1f us/step, per proj %s"
        % (avg_launch_ms * 1e3, achieved, ksum_ms * 1e3, per_proj))

    unfused = None
    if not args.unfused and not args.no_sweep:
        ustack = Stack(args.workload, dev, bits_list=(3,), fused=False)
        ums, _ = time_graph(ustack, 1, 3, max(20, args.steps // 4), 5)
        unfused = {"us_per_step": round(ums * 1e3, 2), "launches_per_step": len(ustack.shapes),
                   "GBps": round(wbytes / (ums * 1e-3) / 1e9, 1),
                   "per_projection_graph": per_call_graph(ustack, 1, 3)}
        log("unfused (one call per projection):", unfused)
        gms, _ = time_graph(ustack, 1, 3, max(20, args.steps // 4), 5,
                            step_fn=lambda: grouped_step(ustack, 1, 3))
        unfused["grouped_launch"] = {"us_per_step": round(gms * 1e3, 2), "launches_per_step": 4 * ustack.layers,
                                     "GBps": round(wbytes / (gms * 1e-3) / 1e9, 1)}
        log("separate weights, shared-stage calls as grouped launches:", unfused["grouped_launch"])
        del ustack
        torch.cuda.empty_cache()

    per_call = per_call_graph(stack, 1, 3)
    log("per call shape (graph of each shape's calls):", per_call)
    dist = replay_distribution(stack, 1, 3)
    log("per-replay step times (W3, M=1):", dist)
    extra = {"us_per_step_graph": round(ms * 1e3, 2), "unfused": unfused, "pct_of_hbm_peak": round(value / HBM_PEAK_GBS * 100, 2),
             "launches_per_step": n_launch, "per_call_graph": per_call,
             "eager_kernel_events": {"sum_us_per_step": round(ksum_ms * 1e3, 2),
                                     "avg_us": round(ksum_ms * 1e3 / n_launch, 3)},
             "per_projection": per_proj,
             "step_us_distribution": dist,
             "wall_s_timed_region": round(wall, 4)}

    if not args.no_sweep:
        sweep = {}
        for bits in (3, 4):
            for M in (1, 4, 8, 16):
                ms_b, _ = time_graph(stack, M, bits, max(20, args.steps // 4), 5)
                sweep["w%d_m%d" % (bits, M)] = {"us": round(ms_b * 1e3, 2),
                                                "GBps": round(stack.weight_bytes(bits) / (ms_b * 1e-3) / 1e9, 1)}
        extra["sweep"] = sweep
        log("sweep", sweep)
        extra["single_1024"] = single_extra(dev)
        log("single 1024 x 1024:", extra["single_1024"])
        # quantize throughput over the whole stack (fp16 read + packed write):
        # all calls captured in one HIP graph (as the linear stack), and the
        # same calls launched eagerly from Python for comparison
        qd = []
        for bits in (3, 4):
            outs = stack.q[bits]

            def quantize_all():
                for i, w in enumerate(stack.fp16):
                    laq.quantize(w, bits, out=outs[i])
            qms = time_calls_graph(quantize_all)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            quantize_all()
            e1.record()
            torch.cuda.synchronize()
            ems = e0.elapsed_time(e1)
            qbytes = stack.weights() * (2 + bytes_per_weight(bits))
            qd.append(("w%d" % bits, {"ms": round(qms, 3), "GBps": round(qbytes / (qms * 1e-3) / 1e9, 1),
                                      "eager_ms": round(ems, 3)}))
        # pack with given parameters (the ones quantize just wrote), W3
        outs = stack.q[3]

        def pack_all():
            for i, w in enumerate(stack.fp16):
                laq.pack(w, outs[i][1], outs[i][2], 3, out=outs[i][0])
        pms = time_calls_graph(pack_all)
        qd.append(("pack_w3", {"ms": round(pms, 3), "GBps": round(stack.weights() * (2 + bytes_per_weight(3)) / (pms * 1e-3) / 1e9, 1)}))
        extra["quantize_stack"] = dict(qd)
        log("quantize", extra["quantize_stack"])
        # unquantized reference: fp16 weights through torch's dense GEMM
        fp = {}
        for M in (1, 16):
            fms = time_fp16_graph(stack, M, max(20, args.steps // 4), 5)
            w3 = sweep["w3_m%d" % M]["us"]
            fp["m%d" % M] = {"us": round(fms * 1e3, 2), "GBps": round(stack.weights() * 2 / (fms * 1e-3) / 1e9, 1),
                             "w3_speedup": round(fms * 1e3 / w3, 3)}
        extra["fp16_dense_torch"] = fp
        log("fp16 dense (torch.mm):", fp)
        if args.workload == "stack4b":
            extra["decode_step_4b"] = decode_step_extra(stack, dev, max(20, args.steps // 4))
            log("decode step:", extra["decode_step_4b"])

    if not args.no_sweep:
        stack.fp16 = None  # free the 4B stack's tensors; its shapes stay for the report
        stack.q = None
        stack.x = None
        stack.y = None
        torch.cuda.empty_cache()
        extra["stack32b"] = stack32b_extra(dev, max(10, args.steps // 10))

    traffic = measured_traffic()
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "stack4b: 36-layer Qwen3-4B-shaped decode-step linear stack "
                               "(q,k,v,o,gate,up,down per layer), W3G128, M=1",
                   "calls_per_layer": "q|k|v, o, gate|up, down (shared-input projections fused)"
                   if stack.fused else "q, k, v, o, gate, up, down",
                   "layers": stack.layers, "linears_per_step": len(stack.shapes), "M": 1, "bits": 3,
                   "group": GROUP, "weights_per_step": stack.weights(),
                   "weight_bytes_per_step": int(round(wbytes))},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None if traffic is None else traffic["hbm_bytes_per_launch"],
                     "algorithmic_bytes_per_launch": int(round(wbytes / len(stack.shapes))),
                     "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                     "kernel": "linear_flat_kernel<3,1,...> (W3G128 GEMV, M=1), all calls of the step"},
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(),
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
