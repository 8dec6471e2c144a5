#!/usr/bin/env python3
"""Selective-recompute prefill benchmark on one MI355X.

One step = one check layer of the selective-recompute prefill
(kvc_blend_prefill_layer) on the 124k-context workload: 16 reused chunks of
7,750 tokens plus a 256-token query chunk (124,256 rows), Llama-3.1-8B
attention shape (32 q heads, 8 kv heads, head size 128, bf16), 15 % of the
reused tokens recomputed.  The step runs every hot-path stage: RoPE
re-positioning of the reused keys, key deviation, top-k selection, scatter
of the recomputed K/V, and sparse-query causal GQA attention.  Inputs are
seeded synthetic tensors (no model weights or datasets), resident in HBM
before timing starts.

Prints one JSON line (see the repository's benchmark contract), including
per-stage times, the attention roofline, a full-causal attention comparison
(every row recomputed, same kernel) and the CPU oracle timed on a bounded
sample of the same workload.

    python bench.py [--steps 20] [--warmup 3] [--config 124k] [--ratio 0.15]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0         # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="124k",
                    choices=["tiny", "4k", "32k", "124k", "124k-tp8", "sep-4k", "qa-32k", "qa-124k", "docs-124k"])
    ap.add_argument("--ratio", type=float, default=0.15)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--stage-reps", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full-causal", action="store_true")
    ap.add_argument("--layouts", default="qa-124k,docs-124k",
                    help="document layouts (zero-K/V separators, many chunks) timed after the headline "
                         "workload; empty for none")
    ap.add_argument("--layers", type=int, default=32,
                    help="also time a prefill of this many layers (0 = skip)")
    ap.add_argument("--layer-reps", type=int, default=2)
    ap.add_argument("--no-layer-share", action="store_true",
                    help="skip the whole-layer measurement (projections + MLP around the attention)")
    ap.add_argument("--pipeline-layers", type=int, default=32,
                    help="layers of the host-to-device pipeline measurement (0: skip)")
    ap.add_argument("--graph-configs", default="tiny,4k,32k",
                    help="small workloads whose check layer is also timed replayed from a HIP graph; "
                         "empty for none")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# --------------------------------------------------------------------------
# inputs: seeded raw draws (workloads) -> device; positional encoding of the
# model's keys/queries applied here with torch (input preparation only)
# --------------------------------------------------------------------------
def make_inputs(w, seed, torch, np):
    import workloads as W
    dev = torch.device("cuda:0")
    t0 = time.time()
    raw = W.draw_raw(w, seed, 0)
    log(f"drew raw tensors in {time.time() - t0:.1f}s")
    N, n_r = w.n_rows, w.n_reused
    j = torch.arange(w.head_dim // 2, dtype=torch.float64, device=dev)
    inv = torch.tensor(w.rope_theta, dtype=torch.float64, device=dev) ** (-(2.0 * j) / w.head_dim)
    local = torch.cat([torch.arange(L, dtype=torch.float64, device=dev) for L in w.chunk_len]
                      + [torch.arange(n_r, N, dtype=torch.float64, device=dev)])
    glob = torch.arange(N, dtype=torch.float64, device=dev)

    def rope_bf16(x_np, pos, extra=None):
        out = torch.empty(x_np.shape, dtype=torch.bfloat16, device=dev)
        step = 16384
        for a in range(0, x_np.shape[0], step):
            x = torch.from_numpy(x_np[a:a + step]).to(dev).to(torch.float64)
            if extra is not None:
                x = x + torch.from_numpy(extra[a:a + step]).to(dev).to(torch.float64)
            ang = pos[a:a + step, None] * inv[None, :]
            c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
            h = w.head_dim // 2
            x1, x2 = x[..., :h], x[..., h:]
            out[a:a + step] = torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], dim=-1).to(torch.bfloat16)
        return out.view(torch.int16)

    def bf16(x_np, extra=None):
        x = torch.from_numpy(x_np).to(dev)
        if extra is not None:
            x = x + torch.from_numpy(extra).to(dev)
        return x.to(torch.bfloat16).view(torch.int16)

    x = dict(k_src=rope_bf16(raw["k_raw"], local), k_fresh=rope_bf16(raw["k_raw"], glob, raw["k_noise"]),
             v_cache=bf16(raw["v"]), v_fresh=bf16(raw["v"], raw["v_noise"]),
             q=rope_bf16(raw["q_raw"], glob))
    del raw
    z = w.zero_rows
    if len(z):
        # separator slots: cached K/V all zero (recomputed K/V as drawn)
        zt = torch.from_numpy(z).to(dev)
        x["k_src"][zt] = 0
        x["v_cache"][zt] = 0
    torch.cuda.synchronize()
    log(f"inputs on device in {time.time() - t0:.1f}s")
    return x


class Timer:
    """HIP events on the stream the library launches on (torch's current stream)."""

    def __init__(self, torch):
        self.torch = torch

    def run(self, fn, reps):
        t = self.torch
        a, b = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
        t.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        t.cuda.synchronize()
        return a.elapsed_time(b) / reps  # ms

    def spread(self, fn, reps):
        """Each call between its own pair of events: median, min and max in ms."""
        t = self.torch
        evs = [(t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)) for _ in range(reps)]
        t.cuda.synchronize()
        for a, b in evs:
            a.record()
            fn()
            b.record()
        t.cuda.synchronize()
        v = sorted(a.elapsed_time(b) for a, b in evs)
        mid = len(v) // 2
        med = v[mid] if len(v) % 2 else 0.5 * (v[mid - 1] + v[mid])
        return {"median": round(med, 4), "min": round(v[0], 4), "max": round(v[-1], 4), "n": len(v)}


def cpu_baseline(w, x, sel_np, dev_np, torch, np):
    """The oracle, as it stands, on a bounded sample of the same workload."""
    import oracle
    from oracle import bf16_to_f64  # noqa: F401
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = cores
    n_r, N = w.n_reused, w.n_rows
    f = oracle.inv_freq(w.head_dim, w.rope_theta)
    row0 = np.concatenate([[0], np.cumsum(w.chunk_len)[:-1]])
    # a1: every reused chunk but the first (which keeps its positions)
    cs = list(range(1, len(w.chunk_len)))
    a, L = int(row0[cs[0]]), int(sum(w.chunk_len[c] for c in cs))
    ks = x["k_src"][a:a + L].cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    sh = oracle.f64_to_bf16(oracle.rope_shift(ks, [w.chunk_len[c] for c in cs], f,
                                              old_pos0=[-a] * len(cs)))
    t_shift = (time.perf_counter() - t) * n_r / L
    # a2: all rows of those chunks
    m = L
    kf = x["k_fresh"][a:a + m].cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    oracle.key_deviation(sh[:m], kf)
    t_dev = (time.perf_counter() - t) * n_r / m
    # a3: the full selection on the deviations of this workload
    k = oracle.recompute_count(w.ratio, n_r)
    t = time.perf_counter()
    oracle.selection(dev_np, k, n_r, N)
    t_sel = time.perf_counter() - t
    # a4: the blend copy of all selected rows (numpy fancy indexing)
    kc = x["k_src"].cpu().numpy().view(np.uint16)
    vc = x["v_cache"].cpu().numpy().view(np.uint16)
    kfa = x["k_fresh"].cpu().numpy().view(np.uint16)
    vfa = x["v_fresh"].cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    kc[sel_np] = kfa[sel_np]
    vc[sel_np] = vfa[sel_np]
    t_scat = time.perf_counter() - t
    # a5: 400 selected queries spread over the positions; the fixed cost of
    # reading K/V into float64 is timed once and not scaled
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([rng.choice(len(sel_np), 392, replace=False),
                                     np.arange(len(sel_np) - 8, len(sel_np))]))
    q_s = x["q"][torch.from_numpy(sel_np[rows]).cuda()].cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    oracle.sparse_query_attention(q_s[:0], sel_np[rows][:0], kc, vc, w.n_q_heads, w.n_kv_heads)
    t_fixed = time.perf_counter() - t
    t = time.perf_counter()
    oracle.sparse_query_attention(q_s, sel_np[rows], kc, vc, w.n_q_heads, w.n_kv_heads)
    t_rows = time.perf_counter() - t - t_fixed
    frac = float((sel_np[rows] + 1).sum()) / float((sel_np + 1).sum())
    t_attn = t_fixed + t_rows / frac
    total_ms = (t_shift + t_dev + t_sel + t_scat + t_attn) * 1e3
    return {
        "value": round(total_ms, 1), "unit": "ms/layer (extrapolated)", "cores": int(blas),
        "host_cores": cores, "kind": "oracle",
        "sample": (f"float64 numpy oracle: shift of {len(cs)} chunks ({L} rows) scaled x{n_r / L:.1f}; exact "
                   f"deviation of {m} rows scaled x{n_r / m:.1f}; full top-k selection and blend copy; "
                   f"attention of {len(rows)} selected queries scaled by sum(p+1) "
                   f"(x{1 / frac:.0f}) plus the one-off float64 conversion of K/V"),
        "stages_s": {"shift": round(t_shift, 2), "deviation": round(t_dev, 2), "select": round(t_sel, 3),
                     "scatter": round(t_scat, 3), "attention": round(t_attn, 1)},
    }


def multi_layer(w, K, L, plan, n_layers, check_at, reps, seed, torch):
    """Time an n_layers prefill on device-resident synthetic layers.

    Layers before `check_at` are fully recomputed (ratio 1, causal), layer
    `check_at` selects, later layers reuse its selection with compact
    recomputed rows.  Every layer has its own cached K/V (adjusted out of
    place, so repetitions do identical work).  Values are seeded Gaussians
    with lognormal channel scales; positional encoding in float32 (input
    preparation only)."""
    dev = torch.device("cuda:0")
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + seed)
    j = torch.arange(D // 2, dtype=torch.float64, device=dev)
    inv = (torch.tensor(w.rope_theta, dtype=torch.float64, device=dev) ** (-(2.0 * j) / D))
    local = torch.cat([torch.arange(c, dtype=torch.float64, device=dev) for c in w.chunk_len]
                      + [torch.arange(n_r, N, dtype=torch.float64, device=dev)])
    glob = torch.arange(N, dtype=torch.float64, device=dev)

    def rope(x, pos):
        ang = (pos[:, None] * inv[None, :]).to(torch.float32)
        c, s_ = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
        a, b = x[..., :D // 2], x[..., D // 2:]
        return torch.cat([a * c - b * s_, b * c + a * s_], dim=-1)

    def scale(h):
        return torch.exp(0.5 * torch.randn((h, D), generator=g, device=dev))

    k_sel = K.kvc_recompute_count(w.ratio, n_r)
    n_sel = k_sel + w.n_query
    sel = torch.empty(n_sel, dtype=torch.int32, device=dev)
    layers = []
    for layer in range(n_layers):
        sk, sv, sq = scale(Hkv), scale(Hkv), scale(Hq)
        k_raw = torch.randn((N, Hkv, D), generator=g, device=dev) * sk
        v = torch.randn((N, Hkv, D), generator=g, device=dev) * sv
        full = layer <= check_at
        rows = N if full else n_sel
        pos = glob if full else glob[:rows]  # compact rows: values only matter for timing
        d = dict(k_src=rope(k_raw, local).to(torch.bfloat16), v=v.to(torch.bfloat16),
                 k_cache=torch.empty((N, Hkv, D), dtype=torch.bfloat16, device=dev),
                 q=rope(torch.randn((rows, Hq, D), generator=g, device=dev) * sq, pos).to(torch.bfloat16),
                 kf=rope(k_raw[:rows] + 0.1 * torch.randn((rows, Hkv, D), generator=g, device=dev), pos).to(torch.bfloat16),
                 vf=(v[:rows] + 0.1 * torch.randn((rows, Hkv, D), generator=g, device=dev)).to(torch.bfloat16),
                 ratio=1.0 if layer < check_at else w.ratio, check=full,
                 ns=N if layer < check_at else n_sel,
                 sel=torch.empty(N, dtype=torch.int32, device=dev) if layer < check_at else sel,
                 out=torch.empty((N if layer < check_at else n_sel, Hq, D), dtype=torch.bfloat16, device=dev))
        del k_raw, v
        layers.append(d)
    wb = K.kvc_blend_workspace(L)
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def run():
        for d in layers:
            K.kvc_blend_prefill_layer(L, plan, d["check"], d["ratio"], d["k_src"], d["k_cache"], d["v"], d["q"],
                                      d["kf"], d["vf"], d["sel"], d["ns"], d["out"], None, ws, wb)

    run()
    torch.cuda.synchronize()
    ms = Timer(torch).run(run, reps)
    del layers
    torch.cuda.empty_cache()
    return ms


def pipeline_run(w, K, L, plan, x, sel, n_layers, reps, torch, timer):
    """Layer-wise pipeline with the chunk caches in pinned host memory (Section 3.4).

    Layer 0 selects, layers 1.. reuse.  Every layer stages the same host
    caches (one pinned copy of the cached K and V, which makes the transfer
    work of every layer real and identical) into its own device caches.
    Timed: compute alone (caches already staged), transfer then compute on
    one stream, the two-stream pipeline (transfer of all layers on a copy
    stream, each layer's computation waiting for its own event), and the
    transfer alone."""
    dev = torch.device("cuda:0")
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    n_sel = sel.numel()
    row_bytes = Hkv * D * 2
    hk = x["k_src"][:n_r].cpu().pin_memory()
    hv = x["v_cache"][:n_r].cpu().pin_memory()
    row0 = [0]
    for c in w.chunk_len[:-1]:
        row0.append(row0[-1] + c)
    # one buffer per tensor laid out like the rows (a loader writes each
    # chunk at its offset); separator chunks point into it as well, so each
    # layer is one copy per tensor, and staging zero-fills their rows
    kp = [hk.data_ptr() + r * row_bytes for r in row0] * n_layers
    vp = [hv.data_ptr() + r * row_bytes for r in row0] * n_layers
    kcs = [torch.empty((N, Hkv, D), dtype=torch.int16, device=dev) for _ in range(n_layers)]
    vcs = [torch.empty((N, Hkv, D), dtype=torch.int16, device=dev) for _ in range(n_layers)]
    idx = sel.long()
    fresh = [(x["q"], x["k_fresh"], x["v_fresh"])] + \
        [(x["q"][idx].contiguous(), x["k_fresh"][idx].contiguous(), x["v_fresh"][idx].contiguous())] * (n_layers - 1)
    out = torch.empty((n_sel, Hq, D), dtype=torch.int16, device=dev)
    wb = K.kvc_blend_workspace(L)
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()
    events = [torch.cuda.Event() for _ in range(n_layers)]
    for e in events:
        e.record(copy)

    def compute(l):
        q, kf, vf = fresh[l]
        K.kvc_blend_prefill_layer(L, plan, l == 0, w.ratio, None, kcs[l], vcs[l], q, kf, vf, sel, n_sel,
                                  out, None, ws, wb)

    def only_compute():
        for l in range(n_layers):
            compute(l)

    def serial():
        for l in range(n_layers):
            K.kvc_stage_layer(L, plan, kp[l * len(row0):(l + 1) * len(row0)], vp[l * len(row0):(l + 1) * len(row0)],
                              kcs[l], vcs[l])
            compute(l)

    def pipelined():
        copy.wait_stream(comp)
        K.kvc_stage_layers(L, plan, n_layers, kp, vp, kcs, vcs, events, stream=copy)
        for l in range(n_layers):
            comp.wait_event(events[l])
            compute(l)

    def only_transfer():
        K.kvc_stage_layers(L, plan, n_layers, kp, vp, kcs, vcs, None)

    res = {}
    # transfer first: the compute-only run needs staged caches (uninitialised
    # memory tends to be zero, which the matrix cores process faster)
    for name, fn in (("transfer_only", only_transfer), ("compute_only", only_compute),
                     ("serial", serial), ("pipelined", pipelined)):
        fn()
        torch.cuda.synchronize()
        res[name] = timer.run(fn, reps)
    moved = 2.0 * n_r * row_bytes * n_layers
    out_d = {"layers": n_layers,
             "workload": f"{w.name}, caches of every layer in pinned host memory "
                         f"({2 * n_r * row_bytes / 1e6:.1f} MB per layer)",
             "pipelined_ms": round(res["pipelined"], 2), "serial_ms": round(res["serial"], 2),
             "compute_only_ms": round(res["compute_only"], 2), "transfer_only_ms": round(res["transfer_only"], 2),
             "h2d_GBps": round(moved / (res["transfer_only"] * 1e-3) / 1e9, 1),
             "exposed_transfer_ms": round(res["pipelined"] - res["compute_only"], 2)}
    log(f"pipeline ({n_layers} layers): pipelined {res['pipelined']:.1f} ms, serial {res['serial']:.1f} ms, "
        f"compute only {res['compute_only']:.1f} ms, transfer only {res['transfer_only']:.1f} ms")
    del kcs, vcs, fresh
    torch.cuda.empty_cache()
    return out_d


def layer_share(w, K, L, plan, x, sel, torch, timer, reps=3):
    """Whole Llama-3.1-8B-shaped layers around the library's attention.

    Random bf16 weights (hidden 4096, 32 q / 8 kv heads of 128, MLP 14336,
    SwiGLU, RMSNorm; weights in the [out, in] layout).  The library runs
    every step: the RMS norms (gathering the selected rows), the projections
    (kvc_projection, with the residual additions of the O and down
    projections fused, in place), the Q/K/V split with RoPE, the gated
    SiLU, and the adjustment, deviation, selection, blend and attention.
    torch's bf16 GEMMs (hipBLASLt) on the same shapes are timed beside the
    library's projections for comparison.  Three layer kinds:
      check: keys projected for every row, the selection, then Q/K/V for
             the selected rows only and the rest of the layer on them;
      reuse: everything for the selected rows only;
      full:  every row, causal attention.
    Also reported: the reuse layer's time per step, and each elementwise
    library kernel's algorithmic bandwidth.  The shares are context for the
    headline, which times the library's path alone."""
    dev = torch.device("cuda:0")
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    Hd, I, eps = Hq * D, 14336, 1e-5
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    bf, i16 = torch.bfloat16, torch.int16

    def weight(a, b):
        return (torch.randn((a, b), generator=g, device=dev) * 0.02).to(bf)

    Wqkv, Wo = weight((Hq + 2 * Hkv) * D, Hd), weight(Hd, Hd)
    Wgu, Wd = weight(2 * I, Hd), weight(Hd, I)
    Wk = Wqkv[Hd:Hd + Hkv * D]          # the K heads' rows (contiguous)
    g1 = (1 + 0.1 * torch.randn(Hd, generator=g, device=dev)).to(bf)
    g2 = (1 + 0.1 * torch.randn(Hd, generator=g, device=dev)).to(bf)
    h_all = torch.randn((N, Hd), generator=g, device=dev).to(bf)
    n_sel = sel.numel()
    k_cache = torch.empty((N, Hkv, D), dtype=i16, device=dev)
    v_cache = x["v_cache"].clone()
    sel_w = torch.empty_like(sel)
    sel_full = torch.empty(N, dtype=torch.int32, device=dev)
    wb = K.kvc_blend_workspace(L)
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)

    def proj(a, n, w_, res=None, out=None):
        """a [n, k] (bf16) times w_^T, w_ [n_out, k]; res added, out may be res."""
        if out is None:
            out = torch.empty((n, w_.shape[0]), dtype=bf, device=dev)
        K.kvc_projection(n, w_.shape[0], w_.shape[1], a, n, None, w_, res, out)
        return out

    def norm(h, n_x, rows, n, gamma, res=None):
        out = torch.empty((n, Hd), dtype=bf, device=dev)
        K.kvc_rms_norm(h, n_x, rows, n, Hd, gamma, eps, out, res)
        return out

    def qkv(y, n, pos, hq=Hq, hk=Hkv, hv=Hkv):
        mk = lambda h: torch.empty((n, h, D), dtype=i16, device=dev) if h else None
        q, k, v = mk(hq), mk(hk), mk(hv)
        K.kvc_qkv_rope(y, n, hq, hk, hv, D, pos, w.rope_theta, q, k, v)
        return q, k, v

    def attend(q, k, v, n, rows, is_check, ratio, k_src):
        out = torch.empty((n, Hq, D), dtype=i16, device=dev)
        K.kvc_blend_prefill_layer(L, plan, is_check, ratio, k_src, k_cache, v_cache, q, k, v, rows, n,
                                  out, None, ws, wb)
        return out

    def rest(h, o, n):
        proj(o.view(bf).reshape(n, Hd), n, Wo, res=h, out=h)
        gu = proj(norm(h, n, None, n, g2), n, Wgu)
        a = torch.empty((n, I), dtype=bf, device=dev)
        K.kvc_swiglu(gu, n, I, a)
        proj(a, n, Wd, res=h, out=h)
        return h

    h_sel = torch.empty((n_sel, Hd), dtype=bf, device=dev)

    def check_layer():
        x_all = norm(h_all, N, None, N, g1)
        _, kf, _ = qkv(proj(x_all, N, Wk), N, None, 0, Hkv, 0)
        K.kvc_select_tokens(L, plan, w.ratio, x["k_src"], k_cache, kf, sel_w, n_sel, ws, wb)
        x_sel = norm(h_all, N, sel_w, n_sel, g1, h_sel)
        q, k, v = qkv(proj(x_sel, n_sel, Wqkv), n_sel, sel_w)
        return rest(h_sel, attend(q, k, v, n_sel, sel_w, 0, w.ratio, None), n_sel)

    def reuse_layer():
        xs = norm(h_sel, n_sel, None, n_sel, g1)
        q, k, v = qkv(proj(xs, n_sel, Wqkv), n_sel, sel)
        return rest(h_sel, attend(q, k, v, n_sel, sel, 0, w.ratio, x["k_src"]), n_sel)

    h_full = torch.empty_like(h_all)

    def full_layer():
        xa = norm(h_all, N, None, N, g1)
        q, k, v = qkv(proj(xa, N, Wqkv), N, None)
        h_full.copy_(h_all)
        return rest(h_full, attend(q, k, v, N, sel_full, 1, 1.0, x["k_src"]), N)

    res = {}
    for name, fn in (("check", check_layer), ("reuse", reuse_layer), ("full", full_layer)):
        fn()
        torch.cuda.synchronize()
        res[name] = timer.run(fn, reps)

    # the reuse layer step by step, on preallocated buffers
    xs, x2 = norm(h_sel, n_sel, None, n_sel, g1), norm(h_sel, n_sel, None, n_sel, g2)
    y = proj(xs, n_sel, Wqkv)
    q, k, v = qkv(y, n_sel, sel)
    o = attend(q, k, v, n_sel, sel, 0, w.ratio, x["k_src"])
    gu = proj(x2, n_sel, Wgu)
    a = torch.empty((n_sel, I), dtype=bf, device=dev)
    h_tmp = h_sel.clone()
    kf_all = torch.empty((N, Hkv, D), dtype=i16, device=dev)
    y_k = proj(norm(h_all, N, None, N, g1), N, Wk)
    x_all = torch.empty((N, Hd), dtype=bf, device=dev)
    y_all = proj(x_all, N, Wqkv)
    q_all, k_all, v_all = qkv(y_all, N, None)
    flop = lambda m, kk, nn: 2.0 * m * kk * nn
    steps = {
        "norm": (lambda: K.kvc_rms_norm(h_sel, n_sel, None, n_sel, Hd, g1, eps, xs), 2 * 2 * n_sel * Hd, None),
        "qkv_gemm": (lambda: proj(xs, n_sel, Wqkv, out=y), None, flop(n_sel, Hd, Wqkv.shape[0])),
        "qkv_rope": (lambda: K.kvc_qkv_rope(y, n_sel, Hq, Hkv, Hkv, D, sel, w.rope_theta, q, k, v),
                     2 * 2 * n_sel * (Hq + 2 * Hkv) * D, None),
        "blend_attention": (lambda: K.kvc_blend_prefill_layer(L, plan, 0, w.ratio, x["k_src"], k_cache, v_cache,
                                                               q, k, v, sel, n_sel, o, None, ws, wb), None, None),
        "o_gemm": (lambda: proj(o.view(bf).reshape(n_sel, Hd), n_sel, Wo, res=h_tmp, out=h_tmp), None,
                   flop(n_sel, Hd, Hd)),
        "norm2": (lambda: K.kvc_rms_norm(h_tmp, n_sel, None, n_sel, Hd, g2, eps, x2), 2 * 2 * n_sel * Hd, None),
        "gate_up_gemm": (lambda: proj(x2, n_sel, Wgu, out=gu), None, flop(n_sel, Hd, 2 * I)),
        "swiglu": (lambda: K.kvc_swiglu(gu, n_sel, I, a), 2 * 3 * n_sel * I, None),
        "down_gemm": (lambda: proj(a, n_sel, Wd, res=h_tmp, out=h_tmp), None, flop(n_sel, I, Hd)),
    }
    # the same four GEMMs (and the check layer's all-rows K projection) in
    # torch / hipBLASLt, for comparison only
    y_k2 = torch.empty_like(y_k)
    torch_gemms = {
        "qkv_gemm": (lambda: torch.matmul(xs, Wqkv.t(), out=y), None, flop(n_sel, Hd, Wqkv.shape[0])),
        "o_gemm": (lambda: h_tmp.addmm_(o.view(bf).reshape(n_sel, Hd), Wo.t()), None, flop(n_sel, Hd, Hd)),
        "gate_up_gemm": (lambda: torch.matmul(x2, Wgu.t(), out=gu), None, flop(n_sel, Hd, 2 * I)),
        "down_gemm": (lambda: h_tmp.addmm_(a, Wd.t()), None, flop(n_sel, I, Hd)),
        "k_all_rows_gemm": (lambda: torch.matmul(x_all, Wk.t(), out=y_k2), None, flop(N, Hd, Hkv * D)),
    }
    extra = {
        "k_all_rows_gemm": (lambda: proj(x_all, N, Wk, out=y_k), None, flop(N, Hd, Hkv * D)),
        "norm_gather_all_rows": (lambda: K.kvc_rms_norm(h_all, N, sel, n_sel, Hd, g1, eps, xs, h_tmp),
                                 3 * 2 * n_sel * Hd, None),
        "norm_all_rows": (lambda: K.kvc_rms_norm(h_all, N, None, N, Hd, g1, eps, x_all), 2 * 2 * N * Hd, None),
        "k_rope_all_rows": (lambda: K.kvc_qkv_rope(y_k, N, 0, Hkv, 0, D, None, w.rope_theta, None, kf_all, None),
                            2 * 2 * N * Hkv * D, None),
        "qkv_rope_all_rows": (lambda: K.kvc_qkv_rope(y_all, N, Hq, Hkv, Hkv, D, None, w.rope_theta, q_all, k_all,
                                                     v_all), 2 * 2 * N * (Hq + 2 * Hkv) * D, None),
    }
    breakdown, kernels, torch_ref = {}, {}, {}
    for table, dest in ((steps, breakdown), (extra, kernels), (torch_gemms, torch_ref)):
        for name, (fn, nbytes, nflop) in table.items():
            fn()
            torch.cuda.synchronize()
            ms = timer.run(fn, max(reps, 5))
            d = {"ms": round(ms, 3)}
            if nbytes:
                d["GB/s"] = round(nbytes / ms / 1e6, 1)
                d["frac_of_8TB/s"] = round(nbytes / ms / 1e6 / 8000.0, 3)
            if nflop:
                d["TFLOP/s"] = round(nflop / ms / 1e9, 1)
            dest[name] = d
    for name in ("norm", "qkv_rope", "norm2", "swiglu"):
        kernels[name] = breakdown[name]
    n_layers = 32
    sel_ttft = res["check"] + (n_layers - 1) * res["reuse"]
    full_ttft = n_layers * res["full"]
    out_d = {"model": "Llama-3.1-8B-shaped layer, random bf16 weights; every step in libkvc (norms, "
                      "projections, RoPE, SwiGLU, selection, blend, attention)",
             "check_layer_ms": round(res["check"], 2), "reuse_layer_ms": round(res["reuse"], 2),
             "full_layer_ms": round(res["full"], 2),
             "attention_share_of_reuse_layer": round(breakdown["blend_attention"]["ms"] / res["reuse"], 3),
             "reuse_layer_steps": breakdown, "elementwise_kernels": kernels,
             "torch_hipblaslt_gemms_for_comparison": torch_ref,
             "elementwise_note": "algorithmic bytes per launch / time; repeated launches on inputs up to 256 MB "
                                 "(the selected rows) may be served partly by the MALL, the all-rows launches "
                                 "(0.5-3 GB) stream from HBM",
             "ttft_32_layers_selective_ms": round(sel_ttft, 1), "ttft_32_layers_full_ms": round(full_ttft, 1),
             "ttft_reduction": round(1.0 - sel_ttft / full_ttft, 3)}
    log(f"whole layers: check {res['check']:.2f} ms, reuse {res['reuse']:.2f} ms, full {res['full']:.2f} ms; "
        f"32-layer TTFT {sel_ttft:.0f} vs {full_ttft:.0f} ms")
    log("reuse layer steps (ms): " + ", ".join(f"{k} {v['ms']}" for k, v in breakdown.items()))
    log("projections, kvc_projection vs torch/hipBLASLt (TFLOP/s): " + ", ".join(
        f"{k} {(breakdown.get(k) or kernels.get(k))['TFLOP/s']} vs {v['TFLOP/s']}" for k, v in torch_ref.items()))
    log("elementwise kernels (fraction of 8 TB/s; inputs up to 256 MB may be served by the MALL): " +
        ", ".join(f"{k} {v.get('frac_of_8TB/s')}" for k, v in kernels.items()))
    del Wqkv, Wo, Wgu, Wd, Wk, h_all, h_full, k_cache, v_cache, y, gu, a, y_k, y_k2, x_all, y_all, q_all, k_all, v_all
    torch.cuda.empty_cache()
    return out_d


def graph_run(name, ratio, seed, reps, K, torch, timer):
    """One check layer of a small workload, launched eagerly through the
    binding and replayed from a HIP graph captured once: at these sizes the
    host's launch work (argument checks, 14-16 kernel launches) is a large
    part of a layer, and a graph replays the same kernels with one submission."""
    import numpy as np
    import workloads as W
    w = W.get(name)
    dev = torch.device("cuda:0")
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    x = make_inputs(w, seed, torch, np)
    L = K.Layout(w.chunk_len, w.n_query, Hq, Hkv, D, w.rope_theta)
    pb = K.kvc_plan_bytes(L)
    plan = torch.empty(pb, dtype=torch.uint8, device=dev)
    plan = K.kvc_plan_upload(L, plan, pb)
    n_sel = K.kvc_recompute_count(ratio, n_r) + w.n_query
    k_cache = torch.empty_like(x["k_src"])
    v_cache = x["v_cache"].clone()
    sel = torch.empty(n_sel, dtype=torch.int32, device=dev)
    out = torch.empty((n_sel, Hq, D), dtype=torch.int16, device=dev)
    lse = torch.empty((n_sel, Hq), dtype=torch.float32, device=dev)
    wb = K.kvc_blend_workspace(L) + K.kvc_attention_workspace(n_sel, Hq, Hkv, D)
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)

    def step():
        K.kvc_blend_prefill_layer(L, plan, 1, ratio, x["k_src"], k_cache, v_cache, x["q"], x["k_fresh"],
                                  x["v_fresh"], sel, n_sel, out, lse, ws, wb)

    step()
    torch.cuda.synchronize()
    eager_ms = timer.run(step, reps)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    g.replay()
    torch.cuda.synchronize()
    graph_ms = timer.run(g.replay, reps)
    res = {"workload": f"{name}: {len(w.chunk_len)} chunks, {N} rows, {Hq} q / {Hkv} kv heads, ratio {ratio}",
           "eager_us": round(eager_ms * 1e3, 1), "graph_us": round(graph_ms * 1e3, 1),
           "speedup": round(eager_ms / graph_ms, 2)}
    log(f"graph {name}: eager {res['eager_us']} us, graph replay {res['graph_us']} us per check layer")
    del g, x, k_cache, v_cache
    torch.cuda.empty_cache()
    return res


def layout_run(name, ratio, seed, steps, reps, K, torch, timer):
    """One check layer on a document layout: whole-layer ms and per-stage ms."""
    import numpy as np
    import workloads as W
    w = W.get(name)
    dev = torch.device("cuda:0")
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    x = make_inputs(w, seed, torch, np)
    L = K.Layout(w.chunk_len, w.n_query, Hq, Hkv, D, w.rope_theta)
    pb = K.kvc_plan_bytes(L)
    plan = torch.empty(pb, dtype=torch.uint8, device=dev)
    plan = K.kvc_plan_upload(L, plan, pb)
    k = K.kvc_recompute_count(ratio, n_r)
    n_sel = k + w.n_query
    k_cache = torch.empty_like(x["k_src"])
    v_cache = x["v_cache"].clone()
    sel = torch.empty(n_sel, dtype=torch.int32, device=dev)
    out = torch.empty((n_sel, Hq, D), dtype=torch.int16, device=dev)
    lse = torch.empty((n_sel, Hq), dtype=torch.float32, device=dev)
    wb = K.kvc_blend_workspace(L)
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)

    def step():
        K.kvc_blend_prefill_layer(L, plan, 1, ratio, x["k_src"], k_cache, v_cache, x["q"], x["k_fresh"],
                                  x["v_fresh"], sel, n_sel, out, lse, ws, wb)

    step()
    layer_ms = timer.run(step, steps)
    sel_np = sel.cpu().numpy().astype(np.int64)
    z = w.zero_rows
    dev_buf = torch.empty(max(n_r, 1), dtype=torch.float64, device=dev)
    tws_b = K.kvc_select_topk_workspace(n_r)
    tws = torch.empty(max(tws_b, 16), dtype=torch.uint8, device=dev)
    sel2 = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
    st = {"shift": timer.run(lambda: K.kvc_rope_shift(L, plan, x["k_src"], k_cache), reps),
          "deviation": timer.run(lambda: K.kvc_kv_deviation(n_r, Hkv, D, k_cache, x["k_fresh"], dev_buf), reps),
          "topk": timer.run(lambda: K.kvc_select_topk(dev_buf, n_r, k, sel2, tws, tws_b), reps),
          "scatter": timer.run(lambda: K.kvc_scatter_rows(sel, n_sel, 0, x["k_fresh"], x["v_fresh"], N, k_cache,
                                                          v_cache, N, Hkv, D), reps),
          "attention": timer.run(lambda: K.kvc_sparse_query_attention(
              x["q"], N, sel, sel, n_sel, k_cache, v_cache, N, Hq, Hkv, D, 0.0, out, lse), reps)}
    elem = n_r * Hkv * D
    flop = 4.0 * Hq * D * float((sel_np + 1).sum())
    res = {"workload": f"{name}: {len(w.chunk_len) // 2} documents, {len(w.chunk_len)} chunks "
                       f"(two-token zero-K/V separators), {N} rows, ratio {ratio}",
           "layer_ms": round(layer_ms, 4),
           "shift_ms": round(st["shift"], 4), "shift_GBps": round(4.0 * elem / (st["shift"] * 1e-3) / 1e9, 1),
           "deviation_ms": round(st["deviation"], 4),
           "deviation_GBps": round((4.0 * elem + 8.0 * n_r) / (st["deviation"] * 1e-3) / 1e9, 1),
           "topk_ms": round(st["topk"], 4), "scatter_ms": round(st["scatter"], 4),
           "attention_ms": round(st["attention"], 3),
           "attention_TFLOPs": round(flop / (st["attention"] * 1e-3) / 1e12, 1),
           "separators_selected": f"{int(np.isin(z, sel_np).sum())}/{len(z)}"}
    log(f"layout {name}: layer {layer_ms:.3f} ms; " + ", ".join(f"{a}={b:.4f}" for a, b in st.items()))
    return res


def measured_traffic(config):
    """HBM bytes per attention launch from the committed rocprofv3 counters
    (FETCH_SIZE + WRITE_SIZE, calibrated against a plain copy), or None if the
    kernel source changed since they were taken or the workload differs."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "attention_traffic_124k.json")
    src = os.path.join(ROOT, "paper_2609_09768_amd", "csrc", "attention.hip")
    if config != "124k" or not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    with open(src, "rb") as fh:
        if hashlib.sha256(fh.read()).hexdigest() != rec.get("kernel_source_sha256"):
            return None
    return int(rec["fetch_bytes"]) + int(rec["write_bytes"])


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the selective-recompute prefill of the paper is a "
              "single-GPU inference path and the library has no multi-GPU mode (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as W
    import paper_2609_09768_amd as K

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    timer = Timer(torch)

    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20)
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty(n, dtype=torch.uint8, device=dev)
        a.fill_(1)
        ms = timer.run(lambda: b.copy_(a), 5)
        print(json.dumps({"copy_probe_bytes": n, "ms": ms, "GBps": 2 * n / ms / 1e6}))
        return

    w = W.get(args.config)
    ratio = args.ratio
    N, n_r, Hq, Hkv, D = w.n_rows, w.n_reused, w.n_q_heads, w.n_kv_heads, w.head_dim
    x = make_inputs(w, args.seed, torch, np)
    L = K.Layout(w.chunk_len, w.n_query, Hq, Hkv, D, w.rope_theta)
    pb = K.kvc_plan_bytes(L)
    plan = torch.empty(pb, dtype=torch.uint8, device=dev)
    plan = K.kvc_plan_upload(L, plan, pb)
    k = K.kvc_recompute_count(ratio, n_r)
    n_sel = k + w.n_query
    k_cache = torch.empty_like(x["k_src"])
    v_cache = x["v_cache"].clone()
    sel = torch.empty(n_sel, dtype=torch.int32, device=dev)
    out = torch.empty((n_sel, Hq, D), dtype=torch.int16, device=dev)
    lse = torch.empty((n_sel, Hq), dtype=torch.float32, device=dev)
    # the layer's workspace plus the attention's optional split workspace
    # (zero at 124k, where the selection fills the GPU)
    awb = K.kvc_attention_workspace(n_sel, Hq, Hkv, D)
    wb = K.kvc_blend_workspace(L) + awb
    ws = torch.empty(max(wb, 16), dtype=torch.uint8, device=dev)
    aws = torch.empty(max(awb, 16), dtype=torch.uint8, device=dev)

    def step():
        K.kvc_blend_prefill_layer(L, plan, 1, ratio, x["k_src"], k_cache, v_cache, x["q"], x["k_fresh"],
                                  x["v_fresh"], sel, n_sel, out, lse, ws, wb)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    t_wall = time.perf_counter()
    ms_per_step = timer.run(step, args.steps)
    t_wall = time.perf_counter() - t_wall
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")

    # stage breakdown, each entry point alone on the same stream
    sel_np = sel.cpu().numpy().astype(np.int64)
    dev_buf = torch.empty(max(n_r, 1), dtype=torch.float64, device=dev)
    tws_b = K.kvc_select_topk_workspace(n_r)
    tws = torch.empty(max(tws_b, 16), dtype=torch.uint8, device=dev)
    sel2 = torch.empty(max(k, 1), dtype=torch.int32, device=dev)
    R = args.stage_reps
    st = {}
    st["shift"] = timer.run(lambda: K.kvc_rope_shift(L, plan, x["k_src"], k_cache), R)
    st["deviation"] = timer.run(lambda: K.kvc_kv_deviation(n_r, Hkv, D, k_cache, x["k_fresh"], dev_buf), R)
    st["topk"] = timer.run(lambda: K.kvc_select_topk(dev_buf, n_r, k, sel2, tws, tws_b), R)
    st["scatter"] = timer.run(lambda: K.kvc_scatter_rows(sel, n_sel, 0, x["k_fresh"], x["v_fresh"], N, k_cache,
                                                         v_cache, N, Hkv, D), R)
    st["attention"] = timer.run(lambda: K.kvc_sparse_query_attention(
        x["q"], N, sel, sel, n_sel, k_cache, v_cache, N, Hq, Hkv, D, 0.0, out, lse, aws, awb), R)
    torch.cuda.synchronize()
    log("stages (ms): " + ", ".join(f"{a}={b:.4f}" for a, b in st.items()))
    # per-launch spread of the layer step and of the attention alone
    spread = {"step_ms": timer.spread(step, args.steps),
              "attention_ms": timer.spread(lambda: K.kvc_sparse_query_attention(
                  x["q"], N, sel, sel, n_sel, k_cache, v_cache, N, Hq, Hkv, D, 0.0, out, lse, aws, awb), R)}
    log(f"spread: {spread}")

    attn_flop = 4.0 * Hq * D * float((sel_np + 1).sum())
    attn_tflops = attn_flop / (st["attention"] * 1e-3) / 1e12
    elem = n_r * Hkv * D
    shift_bytes = 4.0 * elem  # out of place: every reused row read and written
    dev_bytes = 4.0 * elem + 8.0 * n_r
    stages = {
        "shift_ms": round(st["shift"], 4),
        "shift_GBps": round(shift_bytes / (st["shift"] * 1e-3) / 1e9, 1),
        "deviation_ms": round(st["deviation"], 4),
        "deviation_GBps": round(dev_bytes / (st["deviation"] * 1e-3) / 1e9, 1),
        "topk_ms": round(st["topk"], 4),
        "scatter_ms": round(st["scatter"], 4),
        "attention_ms": round(st["attention"], 3),
        "attention_TFLOPs": round(attn_tflops, 1),
        "attention_TFLOP_per_call": round(attn_flop / 1e12, 3),
    }
    full = None
    if not args.no_full_causal:
        pos_all = torch.arange(N, dtype=torch.int32, device=dev)
        out_f = torch.empty((N, Hq, D), dtype=torch.int16, device=dev)
        kf_all, vf_all = x["k_fresh"], x["v_fresh"]
        f_ms = timer.run(lambda: K.kvc_sparse_query_attention(x["q"], N, None, pos_all, N, kf_all, vf_all, N,
                                                              Hq, Hkv, D, 0.0, out_f, None), 2)
        f_flop = 4.0 * Hq * D * N * (N + 1) / 2.0
        full = {"attention_ms": round(f_ms, 2), "TFLOPs": round(f_flop / (f_ms * 1e-3) / 1e12, 1),
                "selective_over_full": round(ms_per_step / f_ms, 4)}
        del out_f
        log(f"full causal attention: {f_ms:.2f} ms")

    multi = None
    if args.layers > 0:
        ml = {}
        for check_at in (0, 1):
            t = time.perf_counter()
            ms = multi_layer(w, K, L, plan, args.layers, check_at, args.layer_reps, args.seed, torch)
            ml[check_at] = ms
            log(f"{args.layers}-layer prefill (check layer {check_at}): {ms:.2f} ms "
                f"({ms / args.layers:.3f} ms/layer), took {time.perf_counter() - t:.1f}s")
        multi = {"layers": args.layers,
                 "check_layer_0": {"ms": round(ml[0], 2), "ms_per_layer": round(ml[0] / args.layers, 4),
                                   "note": "layer 0 selects, layers 1.. reuse"},
                 "check_layer_1": {"ms": round(ml[1], 2), "ms_per_layer": round(ml[1] / args.layers, 4),
                                   "note": "layer 0 fully recomputed (causal), layer 1 selects, 2.. reuse"}}

    share = None
    if not args.no_layer_share and ratio == w.ratio:
        share = layer_share(w, K, L, plan, x, sel, torch, timer)
        share["attention_share_of_reuse_layer"] = round(st["attention"] / share["reuse_layer_ms"], 3)

    pipe = None
    if args.pipeline_layers > 0 and ratio == w.ratio:
        Lz = K.Layout(w.chunk_len, w.n_query, Hq, Hkv, D, w.rope_theta, zero_kv=w.zero_kv_flags)
        plan_z = torch.empty(K.kvc_plan_bytes(Lz), dtype=torch.uint8, device=dev)
        plan_z = K.kvc_plan_upload(Lz, plan_z, plan_z.numel())
        pipe = pipeline_run(w, K, Lz, plan_z, x, sel, args.pipeline_layers, 2, torch, timer)

    cpu = None
    if not args.no_cpu_baseline:
        t = time.perf_counter()
        dev_np = dev_buf.cpu().numpy()
        cpu = cpu_baseline(w, x, sel_np, dev_np, torch, np)
        log(f"cpu baseline took {time.perf_counter() - t:.1f}s")

    layouts = None
    names = [n for n in args.layouts.split(",") if n]
    if names:
        del x, k_cache, v_cache, out, lse
        torch.cuda.empty_cache()
        layouts = {n: layout_run(n, ratio, args.seed, max(args.steps // 2, 1), R, K, torch, timer) for n in names}

    graphs = None
    gnames = [n for n in args.graph_configs.split(",") if n]
    if gnames:
        graphs = {n: graph_run(n, ratio, args.seed, 50, K, torch, timer) for n in gnames}

    line = {
        "metric": "selective-recompute prefill ms/layer + attention TFLOP/s at 124k ctx, 15% ratio",
        "value": round(ms_per_step, 4),
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded lognormal-scaled Gaussian K/V/Q, Llama-3.1-8B shape; no weights)",
        "config": {"workload": (f"{w.name}: {len(w.chunk_len)} chunks x {w.chunk_len[0]}" if not w.zero_kv_chunks else
                                f"{w.name}: {len(w.chunk_len) // 2} documents in {len(w.chunk_len)} chunks (zero-K/V separators)")
                               + f" + {w.n_query}-token query = {N} rows, {Hq} q / {Hkv} kv heads, D {D}, check layer, "
                               f"ratio {ratio}",
                   "n_rows": N, "n_selected": n_sel, "ratio": ratio},
        "attention_tflops": round(attn_tflops, 1),
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 1), "peak": BF16_MFMA_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / BF16_MFMA_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(args.config), "traffic_unit": "bytes/launch",
                     "kernel": "sparse_attn_kernel"},
        "stages": stages,
        "spread": spread,
        # key-range splits the attention may use with the workspace given (none at 124k)
        "attention_key_splits": 1 if awb == 0 else awb // (n_sel * Hq * (D + 1) * 4),
        "full_causal": full,
        "multi_layer": multi,
        "layouts": layouts,
        "graph": graphs,
        "pipeline": pipe,
        "layer_share": share,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
