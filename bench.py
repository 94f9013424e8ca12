#!/usr/bin/env python3
"""Image tokens/s of SSD decoding on one MI355X (gfx950).

A step is one ssd_decode_image call: the whole SSD schedule of one batch of
images (prefix prefill, horizontal runs of 5 tokens with one verify round
each, then every row verified r times and committed), i.e. every verify pass
of the batch through the library's HIP kernels; a commit runs inside the pass
of the verify round that follows it (same decisions, fewer passes).  Inputs
(prompt ids and the draft table) are resident in device memory before the
timed region.

Workload (default): the 8B-class bf16 decoder with grouped KV heads (32
layers, d=4096, 32 query / 8 KV heads of 128, MLP 14336, 32768 image codes of
a 65536-id vocabulary), 256-token random prompts, 64x64 grid, batch 8, greedy
rule, r = 5 verify rounds per row.  Weights N(0, 0.02) from seed 0.  Drafts
are planted left to right before the timed steps (ssd_plant_image, untimed):
each is the decode's own greedy argmax given everything before it, kept with
probability p = 0.6, else another code, so round-1 acceptance is p by
construction (reported beside p).  Under the paper's fixed-round schedule the
pass count, and so tokens/s, does not depend on acceptance; the strict decode
(`strict_sweep`, the 7B 32x32 workload at p = 0.3 / 0.6 / 0.9) is where it does.

Prints one JSON line.  `value` comes from the timed steps, run with plain
launches.  One more step then runs with every GEMM and attention launch timed
by its own dispatch-timestamp HIP events; `roofline` is the dominant kernel
from those events: the tiled GEMM against the dense bf16 MFMA peak when it
carries the projections (more than 128 rows per pass), else the
weight-streaming GEMMs against HBM.  Extra keys: `attention` (the attention
kernel on its own bytes), `verify_pass_positions` (one drafted row verified at
rows 1, H/4, H/2, H-1 beside a one-token pass at the same place, the paper's
protocol), `ar_tokens_per_s_same_kernels` (from those one-token passes),
`verify_step_hbm` (algorithmic bytes of a mid-image verify pass over its
time), `separate_commit` (one pass per plan step), `strict_sweep`,
`attention_at_scale` / `gemm_at_scale` (one layer of the 8B shape at context
4352), `draft_head`, and `cpu_baseline` (the oracle on the host cores).
"""
import argparse
import dataclasses
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
# sources the GEMM kernels are compiled from (traffic summaries name their hash)
GEMM_SRCS = [os.path.join(ROOT, "paper_2606_20543_amd", "csrc", f)
             for f in ("kernels_gemm.hip", "tiles.h", "ssd_internal.h")]
TRAFFIC_FILES = {
    "stream": os.path.join(ROOT, "profiles", "gemm_bf16_1b-24x24_traffic.md"),
    "tiled": os.path.join(ROOT, "profiles", "gemm_tile_8b-64x64-b8_traffic.md"),
}
GEMM_CLASSES = ("qkv", "o_proj", "gate_up", "down", "lm_head")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cfg_of(ssd, shape):
    c = ssd.ssd_model_config()
    c.n_layers, c.d_model, c.n_heads, c.n_kv_heads = shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads
    c.head_dim, c.d_ff, c.vocab = shape.head_dim, shape.d_ff, shape.vocab
    c.img_lo, c.img_hi = shape.img_lo, shape.img_hi
    c.dtype = ssd.SSD_BF16 if shape.dtype == "bf16" else ssd.SSD_F32
    c.rms_eps, c.rope_theta = 1e-5, 10000.0
    return c


def schedule_of(ssd, wl, truncate=0, K=0):
    sc = ssd.ssd_schedule()
    sc.grid_h, sc.grid_w, sc.k_h, sc.h_rounds, sc.k_v, sc.b_rounds, sc.i_rounds = wl.grid, wl.grid, 5, 1, 1, \
        wl.rounds, 0
    sc.rule, sc.top_k, sc.temperature = wl.rule, wl.top_k, wl.temperature
    import synth
    sc.seed = synth.SEED_SAMPLING
    sc.truncate, sc.trunc_block = truncate, K
    return sc


def coins(wl, p):
    """Planting coins of every image position (seed 2: keep flags on stream 1,
    replacement codes on stream 2, as synth.plant draws them)."""
    import synth
    B, H = wl.batch, wl.grid
    n = B * H * H
    keep = (synth.uniform(synth.SEED_DRAFTS, 1, n) < p).astype(np.uint8).reshape(B, H, H)
    repl = synth.randint(synth.SEED_DRAFTS, 2, 0, wl.model.v_img - 1, n).astype(np.int32).reshape(B, H, H)
    return keep, repl


def plant(ssd, model, wl, sc, d_prefix, p):
    """Untimed: the draft table planted left to right by the decode itself."""
    import torch
    keep, repl = coins(wl, p)
    dev = torch.device("cuda:0")
    B, H = wl.batch, wl.grid
    d_tab = torch.zeros((B, H, H), dtype=torch.int32, device=dev)
    d_out = torch.zeros((B, H, H), dtype=torch.int32, device=dev)
    t0 = time.perf_counter()
    st = ssd.ssd_plant_image(model, sc, B, wl.prefix, d_prefix, torch.from_numpy(keep).to(dev),
                             torch.from_numpy(repl).to(dev), d_tab, d_out)
    torch.cuda.synchronize()
    return d_tab, st, time.perf_counter() - t0


def acceptance_of(st, p):
    r1 = st.accepted_round[0] / max(st.proposed_round[0], 1)
    n = max(st.proposed_round[0], 1)
    return {"planted_keep_p": p, "round1": r1, "round1_positions": int(st.proposed_round[0]),
            "round1_sampling_sd": float(np.sqrt(p * (1 - p) / n)) if p is not None else None,
            "all_rounds": st.accepted / max(st.proposed, 1),
            "by_round": [st.accepted_round[j] / st.proposed_round[j] if st.proposed_round[j] else None
                         for j in range(8)]}


def position_timing(ssd, model, shape, prefix, H, W, drafts, reps=50):
    """Verify-pass time at four positions of the image (rows 1, H/4, H/2, H-1):
    `reps` verify rounds of one drafted row (K = W, no commit, so the frontier and
    the pass stay the same), each synchronized and timed by the host clock; the
    same for a one-token pass (an AR step on the same kernels).  Median, p10, p90."""
    B, P = prefix.shape
    rows = sorted({1, H // 4, H // 2, H - 1})
    sess = ssd.ssd_prefill(model, B, P, prefix, P + H * W, W)
    prm = ssd.ssd_verify_params()
    prm.rule, prm.temperature = ssd.SSD_GREEDY, 1.0
    fr = np.zeros(B, np.int32)
    out = {"rows": rows, "K": W, "reps": reps, "ms_median": [], "ms_p10": [], "ms_p90": [],
           "ar_step_ms_median": [], "pass_over_ar_step": []}
    try:
        y = 0
        for row in rows:
            prm.commit, prm.round = 1, 0
            while y < row:  # commit rows up to this one (frontier P + row*W)
                tok = np.ascontiguousarray(drafts[:, y, :].astype(np.int32))
                ssd.ssd_verify_step(sess, W, tok, prm, frontier=fr)
                y += 1
            prm.commit = 0
            for K, key in ((W, "pass"), (1, "ar")):
                ts = []
                for j in range(reps + 3):
                    prm.round = j
                    tok = np.ascontiguousarray(drafts[:, row, :K].astype(np.int32))
                    t0 = time.perf_counter()
                    ssd.ssd_verify_step(sess, K, tok, prm, frontier=fr)  # host outputs: synchronizes
                    ts.append(time.perf_counter() - t0)
                ts = np.array(ts[3:]) * 1e3
                if key == "pass":
                    out["ms_median"].append(float(np.median(ts)))
                    out["ms_p10"].append(float(np.percentile(ts, 10)))
                    out["ms_p90"].append(float(np.percentile(ts, 90)))
                else:
                    out["ar_step_ms_median"].append(float(np.median(ts)))
            out["pass_over_ar_step"].append(out["ms_median"][-1] / out["ar_step_ms_median"][-1])
    finally:
        ssd.ssd_free_session(sess)
    out["timing"] = "host clock around each synchronizing ssd_verify_step call (host token buffers)"
    return out


def verify_pass_bytes(shape, B, K, ctx):
    """Algorithmic HBM bytes of one verify pass of B x K tokens at context ctx
    (committed positions): the weights once (bf16 projections, norm gains and
    the output layer's image rows), the KV cache read, the block's KV written,
    the embedding rows gathered."""
    d, D, L = shape.d_model, shape.head_dim, shape.n_layers
    es = 2 if shape.dtype == "bf16" else 4
    layer = d * (shape.n_heads + 2 * shape.n_kv_heads) * D + shape.n_heads * D * d + 3 * d * shape.d_ff + 2 * d
    weights = es * (L * layer + d * shape.v_img + d)
    kv_tok = L * 2 * shape.n_kv_heads * D * es
    return weights + B * ctx * kv_tok + B * K * kv_tok + B * K * d * es


def separate_rate(ssd, model, sc, B, P, d_prefix, d_drafts, steps):
    """The same decode with one backbone pass per plan step (commit passes not
    run inside the next verify round): the paper's step count."""
    import ctypes
    import torch
    g = ssd.ssd_schedule()
    ctypes.memmove(ctypes.addressof(g), ctypes.addressof(sc), ctypes.sizeof(sc))
    g.separate_commit = 1
    d_out = torch.zeros((B, sc.grid_h, sc.grid_w), dtype=torch.int32, device=torch.device("cuda:0"))
    t0 = time.perf_counter()
    for _ in range(steps):
        st = ssd.ssd_decode_image(model, g, B, P, d_prefix, d_drafts, d_out)
    dt = (time.perf_counter() - t0) / steps
    return {"value": B * sc.grid_h * sc.grid_w / dt, "unit": "image tokens/s", "ms_per_image": dt * 1e3 / B,
            "passes_per_image": st.passes, "ms_per_pass": dt * 1e3 / st.passes, "steps": steps}


def guided_rate(ssd, model, shape, sc, prefix, d_drafts, steps, weight=5.0):
    """Image tokens/s of the same decode with classifier-free guidance (weight 5.0,
    the paper's Janus-Pro setting): every image gets an unconditional twin stream
    with a null prompt (id 0 repeated), so each pass carries twice the rows."""
    import ctypes
    import torch
    B, P = prefix.shape
    g = ssd.ssd_schedule()
    ctypes.memmove(ctypes.addressof(g), ctypes.addressof(sc), ctypes.sizeof(sc))
    g.cfg, g.cfg_weight = 1, weight
    both = np.concatenate([prefix, np.zeros_like(prefix)]).astype(np.int32)
    dev = torch.device("cuda:0")
    d_both = torch.from_numpy(both).to(dev)
    d_out = torch.zeros((B, sc.grid_h, sc.grid_w), dtype=torch.int32, device=dev)
    ssd.ssd_decode_image(model, g, B, P, d_both, d_drafts, d_out)  # warmup (allocates the paired workspace)
    t0 = time.perf_counter()
    for _ in range(steps):
        st = ssd.ssd_decode_image(model, g, B, P, d_both, d_drafts, d_out)
    dt = (time.perf_counter() - t0) / steps
    return {"weight": weight, "value": B * sc.grid_h * sc.grid_w / dt, "unit": "image tokens/s",
            "ms_per_image": dt * 1e3 / B, "passes_per_image": st.passes, "sequences": 2 * B,
            "steps": steps, "unconditional_prompt": "id 0 repeated (null prompt of the same length)"}


def heads_rate(ssd, model, shape, sc, prefix, d_prefix, steps, planted_ms):
    """Image tokens/s of the whole SSD loop with drafts from spatial heads: k_h
    horizontal heads and k_v vertical heads of inner size m = 2d (the paper's
    head size), seeded random weights (no trained heads exist here, so the
    acceptance says nothing about the method).  Drafting needs each committed
    row's states before the next verify round, so no commit shares a pass here;
    the drafting time is taken against the planted decode with the same passes
    (planted_ms)."""
    import torch
    import synth
    B, P = prefix.shape
    d, m = shape.d_model, 2 * shape.d_model
    n = sc.k_h + sc.k_v
    heads = [ssd.ssd_draft_head_init(model, m, synth.draft_head_weights(d, m, seed=10 + j), B * sc.grid_w)
             for j in range(n)]
    try:
        d_out = torch.zeros((B, sc.grid_h, sc.grid_w), dtype=torch.int32, device=torch.device("cuda:0"))
        hh, vh = heads[:sc.k_h], heads[sc.k_h:]
        ssd.ssd_decode_image_heads(model, sc, B, P, d_prefix, hh, vh, d_out)  # warmup
        t0 = time.perf_counter()
        for _ in range(steps):
            st = ssd.ssd_decode_image_heads(model, sc, B, P, d_prefix, hh, vh, d_out)
        dt = (time.perf_counter() - t0) / steps
    finally:
        for h in heads:
            ssd.ssd_free_draft_head(h)
    draft_ms = dt * 1e3 / B - planted_ms
    return {"value": B * sc.grid_h * sc.grid_w / dt, "unit": "image tokens/s", "ms_per_image": dt * 1e3 / B,
            "draft_ms_per_image": draft_ms if draft_ms == draft_ms else None,
            "heads": f"{sc.k_h} horizontal + {sc.k_v} vertical, m = 2d",
            "passes_per_image": st.passes, "steps": steps, "acceptance_random_heads": st.accepted / max(st.proposed, 1)}


def copy_calibration(mib):
    """A plain device-to-device copy of known size, for scaling the PMC byte counters."""
    import torch
    n = mib << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    log(f"[bench] copied {mib} MiB three times (calibration)")


def draft_head_cost(ssd, model, shape, tokens, calls=50):
    """Time the spatial draft head f_phi (Eq. 2) drafting one grid row per call:
    inner size m = 2d (the paper's head size), seeded weights, synthetic hidden
    states.  Not part of `value`: the timed steps verify planted drafts."""
    import torch
    import synth
    d, m, R = shape.d_model, 2 * shape.d_model, tokens.shape[0]
    head = ssd.ssd_draft_head_init(model, m, synth.draft_head_weights(d, m), R)
    try:
        dev = torch.device("cuda:0")
        d_h = torch.from_numpy(synth.hidden_states(R, d)).to(dev)
        d_tok = torch.from_numpy(tokens.astype(np.int32)).to(dev)
        d_dr = torch.zeros(R, dtype=torch.int32, device=dev)
        h_dr = np.zeros(R, np.int32)
        for _ in range(3):
            ssd.ssd_draft_head_run(head, R, d_h, d_tok, h_dr)  # host output: synchronizes
        t0 = time.perf_counter()
        for _ in range(calls - 1):
            ssd.ssd_draft_head_run(head, R, d_h, d_tok, d_dr)
        ssd.ssd_draft_head_run(head, R, d_h, d_tok, h_dr)  # the stream is in order: waits for all
        dt = (time.perf_counter() - t0) / calls
    finally:
        ssd.ssd_free_draft_head(head)
    # bf16 weights read once per call: W0, gain, W1, W3, W2, the final-norm gain and the
    # output layer's image rows; plus the fp32 states in and the embedding rows
    by = 2 * (2 * d * d + d + 3 * m * d + d + shape.v_img * d) + R * d * (4 + 2)
    gbs = by / dt / 1e9
    return {"rows": R, "m": m, "calls": calls, "ms_per_call": dt * 1e3, "bytes_per_call": by,
            "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
            "timing": "host clock over back-to-back calls on the library's stream (launch gaps included)"}


def at_scale(ssd, rounds=5):
    """Kernels at the 8B shape (32 query / 8 KV heads of 128, GQA 4, MLP 14336,
    32768 image codes) with 8 sequences verifying 64-token blocks at context
    4352 (the last row of a 64x64 image after a 256-token prompt: 4288 cached
    positions).  One layer of that model is enough (no kernel depends on the
    others); per-launch events on the library's stream give the kernel times.
    `attention_at_scale`: the attention kernel on its own bytes (the KV read
    and the q/o traffic).  `gemm_at_scale`: the projections of those 512-row
    passes, which run on the tiled GEMM and are bound by the matrix cores:
    algorithmic FLOPs 2*M*N*K against the dense bf16 peak (the two activation
    planes double what the MFMAs issue)."""
    import synth
    shape = dataclasses.replace(synth.M8B, n_layers=1)
    B, K = 8, 64
    P = 4352 - K
    w = synth.weights(shape)
    model = ssd.ssd_init_model(cfg_of(ssd, shape), w)
    del w
    try:
        sess = ssd.ssd_prefill(model, B, P, synth.prompt(shape, B, P), P + K, K)
        try:
            prm = ssd.ssd_verify_params()
            prm.rule, prm.temperature = ssd.SSD_GREEDY, 1.0
            tok = (synth.random_codes(shape, (B, K)) + shape.img_lo).astype(np.int32)
            fr = np.zeros(B, np.int32)
            ssd.ssd_verify_step(sess, K, tok, prm, frontier=fr)  # warm
            ssd.ssd_profile(model, 1)
            ssd.ssd_profile_read(model, reset=True)
            for r in range(rounds):
                prm.round = r + 1
                ssd.ssd_verify_step(sess, K, tok, prm, frontier=fr)
            prof = ssd.ssd_profile_read(model, reset=True)
            ssd.ssd_profile(model, 0)
        finally:
            ssd.ssd_free_session(sess)
    finally:
        ssd.ssd_free_model(model)
    ms, n, by, fl = prof["attention"]
    gbs = by / (ms / 1e3) / 1e9
    att = {"shape": "8B: 32q/8kv heads x 128, batch 8, 64-token blocks, context 4352", "kernel": "attn_qs_kernel",
           "bound": "hbm",
           "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "launches": n,
           "ms_per_launch": ms / n, "bytes_per_launch": by / n, "tflops": fl / (ms / 1e3) / 1e12,
           "timing": "dispatch-timestamp events around each attention launch"}
    classes, tot_f, tot_ms = {}, 0.0, 0.0
    for c in GEMM_CLASSES:
        cms, cn, _, cf = prof[c]
        if not cn:
            continue
        classes[c] = {"ms_per_call": cms / cn, "tflops": cf / (cms / 1e3) / 1e12}
        tot_f += cf
        tot_ms += cms
    tf = tot_f / (tot_ms / 1e3) / 1e12
    gemm = {"shape": "8B projections at M = 512 rows (batch 8 x 64-token blocks)", "kernel": "gemm_tile8_kernel + gemm_tile_kernel",
            "bound": "mfma", "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": tf / MFMA_BF16_PEAK_TFLOPS, "issued_frac": 2 * tf / MFMA_BF16_PEAK_TFLOPS, "classes": classes,
            "timing": "dispatch-timestamp events around each GEMM launch (one per projection per pass)"}
    return {"attention_at_scale": att, "gemm_at_scale": gemm}


def gemm_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SRCS:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kind, workload):
    """HBM bytes per GEMM launch from a committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary; None when the summary is missing, for another workload, or taken
    on a different GEMM source than the one built now."""
    try:
        with open(TRAFFIC_FILES[kind]) as fh:
            kv = dict(l.split(":", 1) for l in fh.read().splitlines() if l.startswith("- ") and ":" in l)
    except (OSError, KeyError):
        return None
    kv = {k[2:].strip(): v.strip() for k, v in kv.items()}
    if kv.get("workload") != workload or kv.get("gemm sources sha256") != gemm_source_hash():
        return None
    try:
        return float(kv["hbm bytes per launch"])
    except (KeyError, ValueError):
        return None


def strict_sweep(ssd, name="7b-32x32", ps=(0.3, 0.6, 0.9), K=32, steps=2):
    """Acceptance-dependent throughput: the strict greedy decode (Sec. 3.3's
    exact contrast case) of the 7B 32x32 workload, blocks of K = 32 (the
    pending token and 31 drafts), drafts planted by the decode itself with keep
    probability p; image tokens/s per p, and greedy AR on the same kernels
    (one-token passes) for reference."""
    import torch
    import synth
    wl = synth.WORKLOADS[name]
    shape, B, P, H = wl.model, wl.batch, wl.prefix, wl.grid
    log(f"[bench] strict sweep {name}: generating weights")
    w = synth.weights(shape)
    model = ssd.ssd_init_model(cfg_of(ssd, shape), w)
    del w
    dev = torch.device("cuda:0")
    res = {"workload": name, "block": K, "batch": B, "grid": f"{H}x{H}", "runs": []}
    try:
        prefix = synth.prompt(shape, B, P)
        d_prefix = torch.from_numpy(prefix.astype(np.int32)).to(dev)
        sc = schedule_of(ssd, wl, truncate=1, K=K)
        d_out = torch.zeros((B, H, H), dtype=torch.int32, device=dev)
        for p in ps:
            d_tab, pst, plant_s = plant(ssd, model, wl, sc, d_prefix, p)
            ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_tab, d_out)  # warm
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                st = ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_tab, d_out)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / steps
            assert st.accepted == pst.accepted and st.passes == pst.passes
            res["runs"].append({"planted_keep_p": p, "value": B * H * H / dt, "unit": "image tokens/s",
                                "ms_per_image": dt * 1e3 / B, "verify_passes": int(st.verify_rounds),
                                "tokens_per_pass": B * H * H / max(st.verify_rounds, 1),
                                "acceptance_tested": st.accepted / max(st.proposed, 1),
                                "drafts_tested": int(st.proposed), "planting_s": plant_s, "steps": steps})
            log(f"[bench] strict p={p}: {res['runs'][-1]['value']:.0f} image tokens/s, "
                f"{st.verify_rounds} passes, acceptance {res['runs'][-1]['acceptance_tested']:.3f}")
        # greedy AR on the same kernels: one-token commit passes at mid-image
        sess = ssd.ssd_prefill(model, B, P, prefix, P + H * H + 1, 1)
        try:
            prm = ssd.ssd_verify_params()
            prm.rule, prm.temperature, prm.commit = ssd.SSD_GREEDY, 1.0, 1
            tok = torch.full((B, 1), shape.img_lo, dtype=torch.int32, device=dev)
            for _ in range(5):
                ssd.ssd_verify_step(sess, 1, tok, prm)
            n = 100
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(n):
                ssd.ssd_verify_step(sess, 1, tok, prm)
            fr = np.zeros(B, np.int32)
            prm.commit = 0
            ssd.ssd_verify_step(sess, 1, np.full((B, 1), shape.img_lo, np.int32), prm, frontier=fr)
            ar_ms = (time.perf_counter() - t0) * 1e3 / (n + 1)
        finally:
            ssd.ssd_free_session(sess)
        res["ar_ms_per_token_pass"] = ar_ms
        res["ar_tokens_per_s_same_kernels"] = B * 1e3 / ar_ms
        for r in res["runs"]:
            r["speedup_vs_ar"] = r["value"] / res["ar_tokens_per_s_same_kernels"]
    finally:
        ssd.ssd_free_model(model)
    return res


def cpu_info():
    model, sockets = None, set()
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name") and model is None:
                    model = line.split(":", 1)[1].strip()
                elif line.startswith("physical id"):
                    sockets.add(line.split(":", 1)[1].strip())
    except OSError:
        pass
    model = model or platform.processor() or "unknown"
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    return {"cpu_model": model, "sockets": max(len(sockets), 1), "logical_cpus": os.cpu_count(),
            "threads": int(threads)}


def cpu_baseline(wl, w, prefix, drafts, passes_per_image, gpu_ms_per_pass):
    """The oracle (numpy float64) on the host cores, on a bounded sample.

    Small workloads (up to 24x24): the whole image of the workload.  Larger ones:
    one verify pass of the workload's shape (B sequences x one W-token row, at
    the first vertical row) through a 2-layer model of the same widths, the
    output layer timed apart; the full model's pass time is the output layer
    plus n_layers times the per-layer time, and image tokens/s that time over
    the image's passes (labelled extrapolated)."""
    from oracle import decode as Dc
    from oracle import model as M
    import synth
    info = cpu_info()
    shape = wl.model
    B, P, H = wl.batch, wl.prefix, wl.grid
    W = H

    def om_of(shp, weights):
        return M.Model(M.Config(shp.n_layers, shp.d_model, shp.n_heads, shp.n_kv_heads, shp.head_dim,
                                shp.d_ff, shp.vocab, shp.img_lo, shp.img_hi, shp.dtype), weights)
    if H <= 24 and shape.n_layers * shape.d_model <= 24 * 2048:
        om = om_of(shape, w)
        codes = drafts - shape.img_lo
        t0 = time.perf_counter()
        tok, st = Dc.decode_image(om, prefix, H, W, codes, rule=wl.rule, seed=3, top_k=wl.top_k, b=wl.rounds)
        dt = time.perf_counter() - t0
        n_tok = B * H * W
        return dict(info, value=n_tok / dt, unit="image tokens/s", cores=info["threads"], kind="oracle",
                    sample=f"prefill + the whole {H}x{W} image ({st['passes']} passes, batch {B}) in {dt:.1f} s",
                    extrapolated=False)
    shp2 = dataclasses.replace(shape, n_layers=2)
    om = om_of(shp2, synth.weights(shp2))
    sess = Dc.prefill(om, prefix, P + 2 * W)
    Dc.commit(sess, drafts[:, 0, :] - shape.img_lo)  # row 0 committed: the first vertical row's context
    t0 = time.perf_counter()
    Dc.verify_round(sess, drafts[:, 1, :] - shape.img_lo, 0, wl.rule, 0, 3, 1.0, wl.top_k)
    t_pass2 = time.perf_counter() - t0
    x = np.random.default_rng(0).standard_normal((B, W, shape.d_model))
    t0 = time.perf_counter()
    M.rms_norm(x, om.final_norm, om.cfg.rms_eps) @ om.lm_img.T
    t_head = time.perf_counter() - t0
    t_layer = max(t_pass2 - t_head, 1e-9) / 2
    t_pass = t_head + shape.n_layers * t_layer
    return dict(info, value=B * H * W / (t_pass * passes_per_image), unit="image tokens/s", cores=info["threads"],
                kind="oracle", extrapolated=True,
                sample=f"one verify pass of {B} x {W} tokens at context {P + W} through a 2-layer model of the "
                       f"same widths ({t_pass2:.2f} s, output layer {t_head:.2f} s), extrapolated to "
                       f"{shape.n_layers} layers ({t_pass:.1f} s per pass) and {passes_per_image} passes per image",
                ms_per_pass=t_pass * 1e3, gpu_speedup_per_pass=t_pass * 1e3 / gpu_ms_per_pass)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="8b-64x64-b8")
    ap.add_argument("--accept-p", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-events", action="store_true", help="skip the per-launch event step")
    ap.add_argument("--forward", choices=("kernels", "persistent"), default="kernels",
                    help="forward pass: one launch per projection/attention, or one cooperative launch per pass "
                         "(blocks of up to 32 tokens)")
    ap.add_argument("--no-draft-head", action="store_true", help="skip the draft-head timing")
    ap.add_argument("--no-positions", action="store_true", help="skip the per-position verify-pass timing")
    ap.add_argument("--no-separate", action="store_true", help="skip the one-pass-per-plan-step timing")
    ap.add_argument("--no-attn-scale", action="store_true", help="skip the kernels at the 8B shape, context 4352")
    ap.add_argument("--no-strict", action="store_true", help="skip the strict-decode sweep (7B 32x32)")
    ap.add_argument("--random-drafts", action="store_true",
                    help="uniform random drafts instead of planting (same passes; for counter runs)")
    ap.add_argument("--cfg", action="store_true", help="also time the decode with classifier-free guidance")
    ap.add_argument("--heads", action="store_true", help="also time the loop drafted by seeded spatial heads")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device copy of this size (PMC byte-counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for {args.gpus}); the verify path shards by "
              "independent images (one process per GPU, each with a full weight replica), so a "
              "multi-GPU figure is that many independent one-GPU runs", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib)
        return

    import torch
    os.environ["SSD_FORWARD"] = args.forward  # read at model creation
    import paper_2606_20543_amd as ssd
    import synth

    t_start = time.perf_counter()
    wl = synth.WORKLOADS[args.workload]
    shape = wl.model
    B, P, H = wl.batch, wl.prefix, wl.grid
    W = H
    p_keep = args.accept_p if args.accept_p is not None else wl.accept_p[len(wl.accept_p) // 2]
    log(f"[bench] workload {wl.name}: generating weights")
    w = synth.weights(shape)
    model = ssd.ssd_init_model(cfg_of(ssd, shape), w)
    prefix = synth.prompt(shape, B, P)
    dev = torch.device("cuda:0")
    d_prefix = torch.from_numpy(prefix.astype(np.int32)).to(dev)
    d_out = torch.zeros((B, H, W), dtype=torch.int32, device=dev)
    sc = schedule_of(ssd, wl)

    if args.random_drafts:
        d_drafts = torch.from_numpy((synth.random_codes(shape, (B, H, W)) + shape.img_lo).astype(np.int32)).to(dev)
        pst = ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_drafts, d_out)
        plant_s, p_keep = 0.0, None
    else:
        log(f"[bench] planting drafts left to right (keep p = {p_keep})")
        d_drafts, pst, plant_s = plant(ssd, model, wl, sc, d_prefix, p_keep)
        log(f"[bench] planted in {plant_s:.1f} s; round-1 acceptance "
            f"{pst.accepted_round[0] / pst.proposed_round[0]:.4f}")
    for i in range(args.warmup):
        ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_drafts, d_out)
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    # timed region: plain launches (per-launch timing adds gaps between kernels)
    ssd.ssd_profile(model, 0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stats = None
    for i in range(args.steps):
        stats = ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_drafts, d_out)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    log(f"[bench] timed {args.steps} steps in {dt:.3f} s")
    assert stats.accepted == pst.accepted and stats.passes == pst.passes, "the planted table did not reproduce"
    # one more step with every GEMM / attention launch timed by its own
    # dispatch-timestamp events (on the library's stream)
    prof = None
    if not args.no_events:
        ssd.ssd_profile(model, 1)
        ssd.ssd_profile_read(model, reset=True)
        ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_drafts, d_out)
        prof = ssd.ssd_profile_read(model, reset=True)
        ssd.ssd_profile(model, 0)
        log("[bench] profiled 1 step")
    if prof is None:
        prof = {c: (0.0, 0, 0.0, 0.0) for c in ssd.PROFILE_CLASSES}

    ms_step = dt * 1000.0 / args.steps
    value = B * H * W / (dt / args.steps)

    def rate(c):
        ms, n, by, fl = prof[c]
        return {"ms_per_launch": ms / max(n, 1), "launches": n, "GB_per_s": by / (ms / 1e3) / 1e9 if ms > 0 else None,
                "TFLOP_per_s": fl / (ms / 1e3) / 1e12 if ms > 0 else None}
    per_class = {c: rate(c) for c in prof}
    t_ms, t_n, t_by, t_fl = prof["tiled_gemm"]
    g_ms = sum(prof[c][0] for c in GEMM_CLASSES)
    g_n = sum(prof[c][1] for c in GEMM_CLASSES)
    g_by = sum(prof[c][2] for c in GEMM_CLASSES)
    s_ms, s_n, s_by = g_ms - t_ms, g_n - t_n, g_by - t_by  # weight-streaming launches
    a_ms, a_n, a_by, a_fl = prof["attention"]
    f_ms, f_n, f_by, _ = prof["forward"]
    timing = ("dispatch-timestamp events (hipExtLaunchKernelGGL) on every launch of one decode step run right "
              "after the timed steps")
    if t_ms >= s_ms and t_ms > 0:
        tf = t_fl / (t_ms / 1e3) / 1e12
        roofline = {"bound": "mfma", "kernel": "gemm_tile8_kernel + gemm_tile_kernel (the tiled GEMMs of the many-row "
                    "passes: gate/up, down and the output layer on 128 x 256 tiles, QKV and the last part of gate/up on 128 x 192, O on 128 x 64)",
                    "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": tf / MFMA_BF16_PEAK_TFLOPS,
                    "traffic": measured_traffic("tiled", wl.name), "traffic_unit": "HBM bytes per launch",
                    "launches": t_n, "ms_per_launch": t_ms / max(t_n, 1), "flops_per_launch": t_fl / max(t_n, 1),
                    "issued_frac": 2 * tf / MFMA_BF16_PEAK_TFLOPS,
                    "issued_note": "every activation is carried as two bf16 planes, so the matrix cores issue twice "
                                   "the algorithmic 2*M*N*K", "timing": timing}
    else:
        gbs = s_by / (s_ms / 1e3) / 1e9 if s_ms > 0 else None
        roofline = {"bound": "hbm", "kernel": "gemm_bf16_kernel + gemm_wide_kernel (weight streaming)",
                    "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS if gbs else None,
                    "traffic": measured_traffic("stream", wl.name), "launches": s_n,
                    "ms_per_launch": s_ms / max(s_n, 1), "bytes_per_launch": s_by / max(s_n, 1), "timing": timing}
    if f_n > 0:
        # the single-launch pass carries the weight stream: it is the kernel the roofline is about
        gbs = f_by / (f_ms / 1e3) / 1e9
        roofline = {"bound": "hbm", "kernel": "fwd_kernel (whole backbone + output layer in one launch)",
                    "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                    "launches": f_n, "ms_per_launch": f_ms / f_n, "bytes_per_launch": f_by / f_n,
                    "timing": "event records around every cooperative launch of the profiled step"}
    a_gbs = a_by / (a_ms / 1e3) / 1e9 if a_ms > 0 else None
    result = {
        "metric": "image tokens/sec (1 GPU) at fixed acceptance; verify-step HBM GB/s % of peak",
        "value": value,
        "unit": "image tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic (random N(0,0.02) weights, random prompt ids, " +
                ("uniform random drafts)" if args.random_drafts else "drafts planted left to right by the decode)"),
        "config": {"workload": wl.name, "batch": B, "prefix": P, "grid": f"{H}x{W}", "rule": wl.rule,
                   "rounds": wl.rounds, "k_h": 5, "k_v": 1, "top_k": wl.top_k, "planted_keep_p": p_keep,
                   "plan_steps_per_image": 1 + 2 * ((W - 1 + 4) // 5) + (H - 1) * (wl.rounds + 1),
                   "passes_per_image": stats.passes, "commit": "run inside the next verify pass where adjacent",
                   "forward": args.forward, "parallelism": "single GPU"},
        "roofline": roofline,
        "attention": {"bound": "hbm", "kernel": "attn_qs_kernel + attn_bf16_kernel", "achieved": a_gbs, "peak": HBM_PEAK_GBS,
                      "unit": "GB/s", "frac": a_gbs / HBM_PEAK_GBS if a_gbs else None, "launches": a_n,
                      "ms_per_launch": a_ms / max(a_n, 1), "bytes_per_launch": a_by / max(a_n, 1),
                      "TFLOP_per_s": a_fl / (a_ms / 1e3) / 1e12 if a_ms > 0 else None},
        "weight_streaming_gemm": {"bound": "hbm", "achieved": s_by / (s_ms / 1e3) / 1e9 if s_ms > 0 else None,
                                  "peak": HBM_PEAK_GBS, "unit": "GB/s", "launches": s_n,
                                  "ms_per_launch": s_ms / max(s_n, 1)},
        "kernel_classes": per_class,
        "acceptance": acceptance_of(stats, p_keep),
        "planting_s": plant_s,
        "verify_ms_per_pass": ms_step / stats.passes,
    }
    if not args.no_positions:
        log("[bench] verify pass at four positions of the image")
        tab = d_drafts.cpu().numpy()
        vp = position_timing(ssd, model, shape, prefix, H, W, tab)
        result["verify_pass_positions"] = vp
        ar_ms = float(np.mean(vp["ar_step_ms_median"]))
        result["ar_tokens_per_s_same_kernels"] = B * 1e3 / ar_ms
        result["ar_note"] = ("one token per sequence per one-token pass, the mean of the four positions' median "
                             "pass times (host clock, synchronizing calls)")
        result["speedup_vs_ar_same_kernels"] = value / result["ar_tokens_per_s_same_kernels"]
        i_mid = vp["rows"].index(H // 2)
        ctx = P + (H // 2) * W
        by = verify_pass_bytes(shape, B, W, ctx)
        gbs = by / (vp["ms_median"][i_mid] / 1e3) / 1e9
        result["verify_step_hbm"] = {"row": H // 2, "context": ctx, "bytes": by, "ms": vp["ms_median"][i_mid],
                                     "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                     "frac": gbs / HBM_PEAK_GBS,
                                     "bytes_note": "weights once + KV read + KV written + embedding rows"}
    if not args.no_separate:
        log("[bench] the same decode with one pass per plan step")
        result["separate_commit"] = separate_rate(ssd, model, sc, B, P, d_prefix, d_drafts, 1)
    if args.cfg:
        log("[bench] the same decode with classifier-free guidance")
        result["cfg"] = guided_rate(ssd, model, shape, sc, prefix, d_drafts, 1)
    if args.heads:
        log("[bench] the whole loop with drafts from spatial heads")
        same = result["separate_commit"]["ms_per_image"] if "separate_commit" in result else float("nan")
        result["heads_decode"] = heads_rate(ssd, model, shape, sc, prefix, d_prefix, 1, same)
    if not args.no_draft_head and shape.dtype == "bf16":
        log("[bench] draft head: one grid row per call")
        row = d_out[0, 0].cpu().numpy().astype(np.int64)
        result["draft_head"] = draft_head_cost(ssd, model, shape, row)
    drafts_host = d_drafts.cpu().numpy()
    ssd.ssd_free_model(model)
    model = None
    if not args.no_attn_scale:
        log("[bench] attention and the tiled GEMMs at the 8B shape, context 4352")
        result.update(at_scale(ssd))
    if not args.no_strict:
        result["strict_sweep"] = strict_sweep(ssd)
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host cores")
        result["cpu_baseline"] = cpu_baseline(wl, w, prefix, drafts_host, stats.passes, ms_step / stats.passes)
    result["bench_wall_s"] = time.perf_counter() - t_start
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
