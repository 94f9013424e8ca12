#!/usr/bin/env python3
"""Image tokens/s of SSD decoding on one MI355X (gfx950).

A step is one ssd_decode_image call: the whole SSD schedule of one batch of
images (prefix prefill, horizontal runs of 5 tokens with one verify round
each, then every row verified r times and committed), i.e. every verify
pass of the image through the library's HIP kernels; a commit runs inside the
pass of the verify round that follows it (same decisions, fewer passes).  Inputs (prompt ids and
planted drafts) are resident in device memory before the timed region.

Workload (default): the 1B-class bf16 decoder (24 layers, d=2048, 16x128
heads, MLP 5632, 16384 image codes), 64-token random prompt, 24x24 grid,
batch 1, greedy rule, r = 2, drafts planted from the backbone's own greedy
AR image with keep-probability 0.6.  Weights N(0, 0.02) from seed 0.

Prints one JSON line (rank 0).  `value` comes from the timed steps, run with
plain launches.  The same number of steps then runs again with every GEMM and
attention launch timed by its own dispatch-timestamp HIP events (per-launch
timing leaves gaps between kernels, so it stays out of the timed steps).
Extra keys: `roofline` (the weight-streaming GEMM kernel, from those events;
with --forward persistent the single-launch forward kernel),
`attention` (the same for the attention kernel), `draft_head` (the spatial
draft head drafting one grid row per call, timed apart from the steps),
`verify_pass_positions` (one drafted row verified at rows 1, H/4, H/2, H-1, 50 reps
each, beside a one-token pass at the same place), `separate_commit` (one pass per
plan step, the paper's step count), `cfg` (the same decode with
classifier-free guidance, weight 5.0), `heads_decode` (the whole loop drafted by
seeded spatial heads instead of planted drafts, and the drafting time per
image), `attention_at_scale` (the attention kernel on its own bytes at the 8B
shape, batch 8, context 4352), `gemm_at_scale` (the tiled GEMM of the same
512-row passes against the dense bf16 MFMA peak), `cpu_baseline` (the oracle
on the host cores on a bounded sample), AR tokens/s on the same kernels.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
# sources the GEMM kernel is compiled from (the traffic summary names their hash)
GEMM_SRCS = [os.path.join(ROOT, "paper_2606_20543_amd", "csrc", f)
             for f in ("kernels_gemm.hip", "tiles.h", "ssd_internal.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_bf16_1b-24x24_traffic.md")


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


def gpu_greedy_ar(ssd, model, shape, prefix, n):
    """Greedy AR decoding through the ABI: one commit pass per token."""
    B, P = prefix.shape
    sess = ssd.ssd_prefill(model, B, P, prefix, P + n + 1, 1)
    out = np.zeros((B, n), np.int64)
    carry = np.zeros((B, shape.v_img), np.float32)
    prm = ssd.ssd_verify_params()
    prm.rule, prm.temperature, prm.commit = ssd.SSD_GREEDY, 1.0, 1
    tok = np.zeros((B, 1), np.int32)
    t0 = time.perf_counter()
    for j in range(n):
        ssd.ssd_get_carry(sess, carry)
        out[:, j] = carry.argmax(axis=1)
        if j + 1 < n:
            tok[:, 0] = out[:, j] + shape.img_lo
            ssd.ssd_verify_step(sess, 1, tok, prm)
    dt = time.perf_counter() - t0
    ssd.ssd_free_session(sess)
    return out, dt


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
                tok = np.ascontiguousarray((drafts[:, y, :] + shape.img_lo).astype(np.int32))
                ssd.ssd_verify_step(sess, W, tok, prm, frontier=fr)
                y += 1
            prm.commit = 0
            for K, key in ((W, "pass"), (1, "ar")):
                ts = []
                for j in range(reps + 3):
                    prm.round = j
                    tok = np.ascontiguousarray((drafts[:, row, :K] + shape.img_lo).astype(np.int32))
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


def separate_rate(ssd, model, sc, B, P, d_prefix, d_drafts, steps):
    """The same decode with one backbone pass per plan step (commit passes not
    run inside the next verify round): the paper's step count."""
    import ctypes
    import torch
    g = ssd.ssd_schedule()
    ctypes.memmove(ctypes.addressof(g), ctypes.addressof(sc), ctypes.sizeof(sc))
    g.separate_commit = 1
    d_out = torch.zeros((B, sc.grid_h, sc.grid_w), dtype=torch.int32, device=torch.device("cuda:0"))
    ssd.ssd_decode_image(model, g, B, P, d_prefix, d_drafts, d_out)
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
    import dataclasses
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
    ms, n, by = prof["attention"]
    gbs = by / (ms / 1e3) / 1e9
    att = {"shape": "8B: 32q/8kv heads x 128, batch 8, 64-token blocks, context 4352", "bound": "hbm",
           "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "launches": n,
           "ms_per_launch": ms / n, "bytes_per_launch": by / n,
           "timing": "dispatch-timestamp events around each attention launch"}
    d, D, M = shape.d_model, shape.head_dim, B * K
    nk = {"qkv": ((shape.n_heads + 2 * shape.n_kv_heads) * D, d), "o_proj": (d, shape.n_heads * D),
          "gate_up": (2 * shape.d_ff, d), "down": (d, shape.d_ff), "lm_head": (shape.v_img, d)}
    classes, tot_f, tot_ms = {}, 0.0, 0.0
    for c, (N, Kd) in nk.items():
        cms, cn, _ = prof[c]
        if not cn:
            continue
        f = 2.0 * M * N * Kd * cn
        classes[c] = {"N": N, "K": Kd, "ms_per_call": cms / cn, "tflops": f / (cms / 1e3) / 1e12}
        tot_f += f
        tot_ms += cms
    tf = tot_f / (tot_ms / 1e3) / 1e12
    gemm = {"shape": "8B projections at M = 512 rows (batch 8 x 64-token blocks)", "kernel": "gemm_tile_kernel",
            "bound": "mfma", "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": tf / MFMA_BF16_PEAK_TFLOPS, "issued_frac": 2 * tf / MFMA_BF16_PEAK_TFLOPS, "classes": classes,
            "timing": "dispatch-timestamp events around each GEMM launch (one per projection per pass)"}
    return {"attention_at_scale": att, "gemm_at_scale": gemm}


def attention_at_scale(ssd):
    """The attention entry of at_scale alone."""
    return at_scale(ssd)["attention_at_scale"]


def gemm_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SRCS:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per GEMM launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary; None when the summary is missing, for another workload, or taken
    on a different GEMM source than the one built now."""
    try:
        with open(TRAFFIC_FILE) as fh:
            kv = dict(l.split(":", 1) for l in fh.read().splitlines() if l.startswith("- ") and ":" in l)
    except OSError:
        return None
    kv = {k[2:].strip(): v.strip() for k, v in kv.items()}
    if kv.get("workload") != workload or kv.get("gemm sources sha256") != gemm_source_hash():
        return None
    try:
        return float(kv["hbm bytes per launch"])
    except (KeyError, ValueError):
        return None


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


def cpu_baseline(wl, w, prefix, drafts):
    """The oracle (numpy float64) on the host cores: the whole image of the
    workload (up to 24 rows), then one verify pass of a drafted row at rows 1,
    H/4, H/2 and H-1 (the rows before each committed first), as the GPU's
    per-position timing does."""
    from oracle import decode as Dc
    from oracle import model as M
    shape = wl.model
    om = M.Model(M.Config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                          shape.d_ff, shape.vocab, shape.img_lo, shape.img_hi, shape.dtype), w)
    rows = min(wl.grid, 24)  # the whole 24x24 image: about 10-20 s of host work on the 1B workload
    t0 = time.perf_counter()
    tok, st = Dc.decode_image(om, prefix, rows, wl.grid, drafts[:, :rows, :], rule=wl.rule, seed=3,
                              top_k=wl.top_k, b=wl.rounds)
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count()
    n_tok = prefix.shape[0] * rows * wl.grid
    H = W = wl.grid
    pos_rows = sorted({1, H // 4, H // 2, H - 1})
    pos_ms = []
    if rows == H:
        sess = Dc.prefill(om, prefix, prefix.shape[1] + H * W)
        y = 0
        for r in pos_rows:
            while y < r:
                Dc.commit(sess, tok[:, y, :])
                y += 1
            t1 = time.perf_counter()
            Dc.verify_round(sess, drafts[:, r, :], 0, wl.rule, 0, 3, 1.0, wl.top_k)
            pos_ms.append((time.perf_counter() - t1) * 1e3)
    return {"value": n_tok / dt, "unit": "image tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"prefill + rows 0-{rows - 1} of the {wl.grid}x{wl.grid} image ({st['passes']} passes, "
                      f"batch {prefix.shape[0]}, {n_tok} tokens) in {dt:.1f} s",
            "verify_pass_positions": {"rows": pos_rows if pos_ms else [], "ms": pos_ms,
                                      "note": "one verify pass of a drafted row at each position, host clock"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="1b-24x24")
    ap.add_argument("--accept-p", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ar", action="store_true", help="also time greedy AR decoding (one pass per token)")
    ap.add_argument("--no-events", action="store_true", help="time without the per-launch event hook")
    ap.add_argument("--forward", choices=("kernels", "persistent"), default="kernels",
                    help="forward pass: one launch per projection/attention, or one cooperative launch per pass "
                         "(blocks of up to 32 tokens)")
    ap.add_argument("--no-draft-head", action="store_true", help="skip the draft-head timing")
    ap.add_argument("--no-positions", action="store_true", help="skip the per-position verify-pass timing")
    ap.add_argument("--no-cfg", action="store_true", help="skip the guided (CFG) decode timing")
    ap.add_argument("--no-separate", action="store_true", help="skip the one-pass-per-plan-step timing")
    ap.add_argument("--no-heads", action="store_true", help="skip the head-drafted decode timing")
    ap.add_argument("--no-attn-scale", action="store_true", help="skip the attention timing at the 8B shape")
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

    wl = synth.WORKLOADS[args.workload]
    shape = wl.model
    B, P, H = wl.batch, wl.prefix, wl.grid
    W = H
    p_keep = args.accept_p if args.accept_p is not None else wl.accept_p[len(wl.accept_p) // 2]
    log(f"[bench] workload {wl.name}: generating weights")
    w = synth.weights(shape)
    cfg = cfg_of(ssd, shape)
    model = ssd.ssd_init_model(cfg, w)
    prefix = synth.prompt(shape, B, P)

    dev = torch.device("cuda:0")
    d_prefix = torch.from_numpy(prefix.astype(np.int32)).to(dev)
    d_out = torch.zeros((B, H, W), dtype=torch.int32, device=dev)
    sc = ssd.ssd_schedule()
    sc.grid_h, sc.grid_w, sc.k_h, sc.h_rounds, sc.k_v, sc.b_rounds, sc.i_rounds = H, W, 5, 1, 1, wl.rounds, 0
    sc.rule, sc.top_k, sc.temperature, sc.seed = wl.rule, wl.top_k, wl.temperature, synth.SEED_SAMPLING

    # Target image: the image one decode commits from random drafts (with a
    # fixed number of rounds the committed image depends on the drafts, so
    # the timed decode, whose drafts keep each target token with probability
    # p_keep (else another code), need not commit it again).  Tokens/s does
    # not depend on the drafts: the pass count is fixed by the schedule.
    log("[bench] target decode (random drafts)")
    d_rand = torch.from_numpy((synth.random_codes(shape, (B, H, W)) + shape.img_lo).astype(np.int32)).to(dev)
    ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_rand, d_out)
    target = d_out.cpu().numpy().astype(np.int64) - shape.img_lo
    drafts = synth.plant(target, p_keep, shape.v_img)
    d_drafts = torch.from_numpy((drafts + shape.img_lo).astype(np.int32)).to(dev)

    ar_rate = None
    if args.ar:
        log("[bench] greedy AR on the GPU (one commit pass per token)")
        ar, ar_dt = gpu_greedy_ar(ssd, model, shape, prefix, H * W)
        ar_rate = B * H * W / ar_dt

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
    # profiled region: the same steps again, every GEMM / attention launch
    # timed by its own dispatch-timestamp events (on the library's stream)
    prof = None
    if not args.no_events:
        ssd.ssd_profile(model, 1)
        ssd.ssd_profile_read(model, reset=True)
        torch.cuda.synchronize()
        tp = time.perf_counter()
        for i in range(args.steps):
            ssd.ssd_decode_image(model, sc, B, P, d_prefix, d_drafts, d_out)
        torch.cuda.synchronize()
        tp = time.perf_counter() - tp
        prof = ssd.ssd_profile_read(model, reset=True)
        ssd.ssd_profile(model, 0)
        log(f"[bench] profiled {args.steps} steps in {tp:.3f} s")

    ms_step = dt * 1000.0 / args.steps
    value = B * H * W / (dt / args.steps)
    classes = ("qkv", "o_proj", "gate_up", "down", "lm_head", "attention", "forward")
    if prof is None:
        prof = {c: (0.0, 0, 0.0) for c in classes}
    f_ms, f_n, f_bytes = prof["forward"]
    f_gbs = f_bytes / (f_ms / 1000.0) / 1e9 if f_ms > 0 else None
    gemm = [prof[c] for c in classes[:5]]
    g_ms = sum(x[0] for x in gemm)
    g_n = sum(x[1] for x in gemm)
    g_bytes = sum(x[2] for x in gemm)
    g_gbs = g_bytes / (g_ms / 1000.0) / 1e9 if g_ms > 0 else None
    a_ms, a_n, a_bytes = prof["attention"]
    a_gbs = a_bytes / (a_ms / 1000.0) / 1e9 if a_ms > 0 else None
    per_class = {c: {"ms_per_launch": prof[c][0] / max(prof[c][1], 1), "launches": prof[c][1],
                     "GB_per_s": prof[c][2] / (prof[c][0] / 1000.0) / 1e9 if prof[c][0] > 0 else None}
                 for c in prof}
    acc = stats.accepted / max(stats.proposed, 1)

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
        "data": "synthetic (random N(0,0.02) weights, random prompt ids, planted drafts)",
        "config": {"workload": wl.name, "batch": B, "prefix": P, "grid": f"{H}x{W}", "rule": wl.rule,
                   "rounds": wl.rounds, "k_h": 5, "k_v": 1, "top_k": wl.top_k, "planted_keep_p": p_keep,
                   "plan_steps_per_image": 1 + 2 * ((W - 1 + 4) // 5) + (H - 1) * (wl.rounds + 1),
                   "passes_per_image": stats.passes, "commit": "run inside the next verify pass where adjacent",
                   "forward": args.forward, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "gemm_bf16_kernel + gemm_wide_kernel (QKV/O/gate-up/down/LM-head weight streaming)",
                     "achieved": g_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": g_gbs / HBM_PEAK_GBS if g_gbs else None,
                     "traffic": measured_traffic(wl.name), "launches": g_n, "ms_per_launch": g_ms / max(g_n, 1),
                     "bytes_per_launch": g_bytes / max(g_n, 1),
                     "timing": "dispatch-timestamp events (hipExtLaunchKernelGGL) on every launch of the profiled "
                               "region, which repeats the timed steps right after them"},
        "forward_launch": {"bound": "hbm", "kernel": "fwd_kernel (whole backbone + output layer in one launch)",
                           "achieved": f_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": f_gbs / HBM_PEAK_GBS if f_gbs else None, "launches": f_n,
                           "ms_per_launch": f_ms / max(f_n, 1), "bytes_per_launch": f_bytes / max(f_n, 1)},
        "attention": {"bound": "hbm", "achieved": a_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                      "frac": a_gbs / HBM_PEAK_GBS if a_gbs else None, "launches": a_n,
                      "ms_per_launch": a_ms / max(a_n, 1)},
        "kernel_classes": per_class,
        "acceptance": acc,
        "verify_ms_per_pass": ms_step / stats.passes,
        "ar_tokens_per_s_same_kernels": ar_rate,
        "speedup_vs_ar_same_kernels": (value / ar_rate) if ar_rate else None,
    }
    if not args.no_positions:
        log("[bench] verify pass at four positions of the image")
        result["verify_pass_positions"] = position_timing(ssd, model, shape, prefix, H, W, drafts)
    if not args.no_separate:
        log("[bench] the same decode with one pass per plan step")
        result["separate_commit"] = separate_rate(ssd, model, sc, B, P, d_prefix, d_drafts, args.steps)
    if not args.no_cfg:
        log("[bench] the same decode with classifier-free guidance")
        result["cfg"] = guided_rate(ssd, model, shape, sc, prefix, d_drafts, args.steps)
    if not args.no_heads:
        log("[bench] the whole loop with drafts from spatial heads")
        same_passes = result["separate_commit"]["ms_per_image"] if "separate_commit" in result else None
        result["heads_decode"] = heads_rate(ssd, model, shape, sc, prefix, d_prefix, args.steps,
                                            same_passes if same_passes is not None else float("nan"))
    if not args.no_draft_head and shape.dtype == "bf16":
        log("[bench] draft head: one grid row per call")
        result["draft_head"] = draft_head_cost(ssd, model, shape, target[0, 0] + shape.img_lo)
    ssd.ssd_free_model(model)
    model = None
    if not args.no_attn_scale:
        log("[bench] attention and the tiled GEMMs at the 8B shape, context 4352")
        result.update(at_scale(ssd))
    if f_n > 0:
        # the single-launch pass carries the weight stream: it is the kernel the roofline is about
        result["roofline"] = dict(result["forward_launch"], traffic=None,
                                  timing="event records around every cooperative launch of the profiled region")
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host cores")
        result["cpu_baseline"] = cpu_baseline(wl, w, prefix, drafts)
        vp = result.get("verify_pass_positions")
        cp = result["cpu_baseline"]["verify_pass_positions"]
        if vp and cp["ms"] and cp["rows"] == vp["rows"]:
            cp["gpu_speedup"] = [c / g for c, g in zip(cp["ms"], vp["ms_median"])]
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
