"""Benchmark of the ISM attention hot path on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                [--only all|step|gqa|bwd|cache|expansion|latency|decode_groups]
                [--calibrate-copy]

A step is one training pass of the attention hot path over one batch of
workload 4, the largest training configuration (4 dialogues x 8192 tokens,
16 turns each, 32 heads, head_dim 128, bf16): the visibility prep, the
forward (which produces the LSE the backward needs) and the backward.
``value`` is the useful (unmasked) TFLOP/s of that step: 4*d FLOPs per
visible (row, key) pair and query head for the forward, 10*d for the
backward; ``tokens_per_s`` gives the same step as packed tokens per second.
``roofline`` is the step's backward, the dominant part (its launches timed
together with HIP events on the launch stream, useful FLOPs only).

The other paths are measured on their own workloads and reported under
``paths``: the forward and the training step of workload 1 (8 x 4096), the
grouped-KV forward (workload 2, 2 x 16384, 32/8 heads), the cached prefill and the decode stream (workload
3, dense and paged, with draft verification, 2-D positions and the measured
streaming-read ceiling), and the decode step with 1, 4, 6 and 8 query heads
per KV head (32 dialogues at position 8192, 8 KV heads).

Two comparisons from the paper ride along under ``paths``: the training cost
of the prefix mask's sample expansion against ISM's single pass over the same
dialogues (Sec. 1), and the per-turn latency experiment of Sec. 3.6 (ISM,
causal and prefix masks; time to first token and per output token) at the
level of one attention layer.

``cpu_baseline`` times the fp64 oracle (test infrastructure, as it stands) on
the host cores, on bounded samples: the step of workload 4 (forward and
backward of some (dialogue, head) pairs) as the headline figure, and the
forwards of workloads 1 and 2 and the cache path of workload 3 (one-shot
reference rows, then 16 stepwise decode steps) beside it.

``--only gqa|bwd|cache|expansion|latency|decode_groups`` measures that one path alone (for
per-kernel profiles of one workload) and prints a JSON line with ``paths``
only; ``--only step`` runs the headline step alone.

The last line of stdout is one JSON object; everything else goes to stderr.

``roofline.traffic`` (HBM bytes per launch of the backward) comes from the
FETCH_SIZE / WRITE_SIZE counter runs recorded in
``profiles/traffic_bwd_4x8192_h32_d128.json``, scaled by what the same
counters read for a plain copy of known size (``--calibrate-copy`` runs that
copy); it is reported only while the kernel sources hash to the value
recorded with the counters, else null.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("ISM attention useful TFLOP/s (fwd, bwd) and % bf16 MFMA peak; "
          "decode HBM GB/s")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_bwd_4x8192_h32_d128.json")
COPY_BYTES = 1 << 30  # --calibrate-copy: bytes read (and written) per copy
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense
PEAK_HBM_GBS = 8000.0
WARM_MS = 200.0      # warmup floor of the paths' measurements (Timer.run)
LAT_WARM_MS = 20.0   # the same for the latency experiment's short launches


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def visible_pairs(segs):
    """Useful (row, key) pairs per query head under the ISM bound: a row of a
    query segment [a, c) sees c - s_b keys, an answer row j sees j - s_b + 1."""
    tot = 0
    cu, cs, fl = segs.cu_seqlens, segs.cu_segs, segs.seg_is_query
    b = 0
    for g in range(len(fl)):
        a, c = int(cs[g]), int(cs[g + 1])
        while not (cu[b] <= a < cu[b + 1]):
            b += 1
        s = int(cu[b])
        n = c - a
        if fl[g]:
            tot += n * (c - s)
        else:
            tot += (a - s + 1 + c - s) * n // 2
    return tot


def dev(bits):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to("cuda")


class Timer:
    """HIP-event timing on torch's current stream (where the ops launch)."""

    def __init__(self):
        import torch
        self.torch = torch
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def run(self, fn, reps, warmup, warm_ms=0.0):
        """Mean ms of ``reps`` calls after ``warmup`` untimed calls and, with
        ``warm_ms``, further untimed calls until that much time has passed
        (after an idle stretch, such as a host-to-device upload, the clock
        needs some tens of ms of work to ramp back up)."""
        for _ in range(warmup):
            fn()
        self.torch.cuda.synchronize()
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < warm_ms:
            fn()
            self.torch.cuda.synchronize()
        self.a.record()
        for _ in range(reps):
            fn()
        self.b.record()
        self.torch.cuda.synchronize()
        return self.a.elapsed_time(self.b) / reps


def device_info():
    """Name, compute units and maximum engine clock of the gfx950 agent, as
    rocminfo reports them (run as a child process; None if unavailable)."""
    import subprocess
    exe = "/opt/rocm/bin/rocminfo"
    try:
        out = subprocess.run([exe], capture_output=True, text=True, timeout=30).stdout
    except (OSError, subprocess.SubprocessError):
        return None
    for agent in out.split("Agent ")[1:]:
        if "gfx950" not in agent:
            continue
        info = {}
        for line in agent.splitlines():
            key, _, val = line.strip().partition(":")
            val = val.strip()
            if key == "Name" and "arch" not in info:
                info["arch"] = val
            elif key == "Marketing Name" and val and "name" not in info:
                info["name"] = val
            elif key == "Compute Unit" and "compute_units" not in info:
                info["compute_units"] = int(val)
            elif key == "Max Clock Freq. (MHz)" and "max_clock_mhz" not in info:
                info["max_clock_mhz"] = int(val)
        info.update(_versions())
        return info
    return None


def _versions():
    """ROCm (the installed release), HIP and torch versions."""
    import torch
    v = {"torch": torch.__version__, "hip": torch.version.hip}
    try:
        with open("/opt/rocm/.info/version") as f:
            v["rocm"] = f.read().strip()
    except OSError:
        pass
    return v


def bench_training(w, timer, steps, warmup, with_bwd):
    from paper_2408_00539_amd import ops
    import torch
    segs = ops.Segments.from_host(w.segs.cu_seqlens, w.segs.cu_segs,
                                  w.segs.seg_is_query)
    q, k, v = dev(w.q), dev(w.k), dev(w.v)
    pairs = visible_pairs(w.segs)
    f_fwd = 4 * w.d * w.hq * pairs
    f_bwd = 10 * w.d * w.hq * pairs
    res = {"visible_pairs_per_head": pairs}
    T = int(w.segs.total)
    o, lse = ops.fwd(q, k, v, segs, w.scale)
    ms_fwd = timer.run(lambda: ops.fwd(q, k, v, segs, w.scale), steps, warmup,
                       WARM_MS)
    res["fwd"] = {"ms": ms_fwd, "tflops": f_fwd / ms_fwd / 1e9,
                  "frac_peak": f_fwd / ms_fwd / 1e9 / PEAK_BF16_TFLOPS,
                  "flop": f_fwd, "tokens_per_s": T / ms_fwd * 1e3}
    if with_bwd:
        do = dev(w.do) if w.do is not None else torch.randn_like(q)
        ms_bwd = timer.run(lambda: ops.bwd(q, k, v, o, lse, do, segs, w.scale),
                           steps, warmup, WARM_MS)
        res["bwd"] = {"ms": ms_bwd, "tflops": f_bwd / ms_bwd / 1e9,
                      "frac_peak": f_bwd / ms_bwd / 1e9 / PEAK_BF16_TFLOPS,
                      "flop": f_bwd, "tokens_per_s": T / ms_bwd * 1e3}

        def step():
            o2, l2 = ops.fwd(q, k, v, segs, w.scale)
            ops.bwd(q, k, v, o2, l2, do, segs, w.scale)
        ms_step = timer.run(step, steps, warmup)
        res["step"] = {"ms": ms_step, "flop": f_fwd + f_bwd,
                       "tokens_per_s": T / ms_step * 1e3}
    else:
        res["step"] = {"ms": ms_fwd, "flop": f_fwd, "tokens_per_s": T / ms_fwd * 1e3}
    return res


def bench_cache(w, timer, reps, warmup):
    from paper_2408_00539_amd import ops
    import torch
    B = len(w.new_lens)
    Kc, Vc = dev(w.k_cache), dev(w.v_cache)
    lens = torch.full((B,), w.hist_len, dtype=torch.int32, device="cuda")
    cu = torch.from_numpy(w.cu_new).cuda()
    qn, kn, vn = dev(w.q_new), dev(w.k_new), dev(w.v_new)
    mx = int(w.new_lens.max())
    L = w.new_lens.astype(np.int64)
    ms_pf = timer.run(lambda: ops.prefill_cached(qn, kn, vn, Kc, Vc, lens, cu,
                                                 mx, w.scale), reps, warmup, WARM_MS)
    f_pf = 4 * w.d * w.hq * float(np.sum(L * (w.hist_len + L)))
    b_pf = 2 * w.hkv * w.d * 2 * float(np.sum(w.hist_len + L))
    out = {"prefill_cached": {
        "ms": ms_pf, "tflops": f_pf / ms_pf / 1e9,
        "frac_peak_mfma": f_pf / ms_pf / 1e9 / PEAK_BF16_TFLOPS,
        "kv_gbs": b_pf / ms_pf / 1e6,
        "bound_ms": max(f_pf / PEAK_BF16_TFLOPS / 1e9, b_pf / PEAK_HBM_GBS / 1e6),
        "flop": f_pf, "kv_bytes": b_pf,
        "new_tokens_per_s": float(np.sum(L)) / ms_pf * 1e3}}
    out["prefill_cached"]["frac_of_bound"] = out["prefill_cached"]["bound_ms"] / ms_pf

    qd, kd, vd = dev(w.q_dec), dev(w.k_dec), dev(w.v_dec)
    pos0 = lens + torch.from_numpy(w.new_lens).cuda()
    ws = torch.empty(ops.workspace_size(ops.ISM_OP_DECODE, B, 0, w.cache_cap,
                                        w.hq, w.hkv, w.d, 0),
                     dtype=torch.uint8, device="cuda")

    def turn():
        pos = pos0.clone()
        for t in range(w.steps):
            ops.decode(qd[t], kd[t], vd[t], Kc, Vc, pos, 0, w.scale,
                       workspace=ws)
            pos += 1
    ms_turn = timer.run(turn, max(1, reps // 4), 1, WARM_MS)
    keys = float(np.sum([np.sum(w.hist_len + L + t + 1) for t in range(w.steps)]))
    b_dec = 2 * w.hkv * w.d * 2 * keys
    out["decode"] = {"steps": w.steps, "ms_per_step": ms_turn / w.steps,
                     "gbs": b_dec / ms_turn / 1e6,
                     "frac_peak_hbm": b_dec / ms_turn / 1e6 / PEAK_HBM_GBS,
                     "bytes": b_dec, "bytes_per_step": b_dec / w.steps,
                     "tokens_per_s": B * w.steps / ms_turn * 1e3,
                     "traffic_per_step": recorded_decode_traffic()}
    # per-step spread: one more turn with an event pair around every step
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(w.steps)]
    pos = pos0.clone()
    for t in range(w.steps):
        ev[t][0].record()
        ops.decode(qd[t], kd[t], vd[t], Kc, Vc, pos, 0, w.scale, workspace=ws)
        ev[t][1].record()
        pos += 1
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) for a, b in ev)
    out["decode"]["step_ms_min"] = per[0]
    out["decode"]["step_ms_median"] = per[len(per) // 2]
    out["decode"]["step_ms_max"] = per[-1]
    out["read_ceiling"] = read_ceiling(timer)
    out["decode"]["frac_of_read_ceiling"] = out["decode"]["gbs"] / out["read_ceiling"]["gbs"]

    # the same turn through a paged cache: pages of 256 positions scattered
    # over a shuffled pool, one block table row per dialogue
    ps = 256
    mp = w.cache_cap // ps
    npages = B * mp + 64
    g = torch.Generator(device="cpu").manual_seed(1234)
    table = torch.randperm(npages, generator=g)[:B * mp].to(torch.int32).view(B, mp).cuda()

    def to_pages(c):
        pool = torch.zeros((npages, w.hkv, ps, w.d), dtype=c.dtype, device=c.device)
        pool[table.view(-1).long()] = (c.view(B, w.hkv, mp, ps, w.d).permute(0, 2, 1, 3, 4)
                                       .reshape(B * mp, w.hkv, ps, w.d))
        return pool
    Kp, Vp = to_pages(Kc), to_pages(Vc)
    ms_pp = timer.run(lambda: ops.prefill_paged(qn, kn, vn, Kp, Vp, table, lens, cu, mx,
                                                True, w.scale), reps, warmup, WARM_MS)
    out["prefill_paged"] = {"ms": ms_pp, "page_size": ps,
                            "tflops": f_pf / ms_pp / 1e9,
                            "vs_dense": ms_pf / ms_pp}

    def turn_paged():
        pos = pos0.clone()
        for t in range(w.steps):
            ops.decode_paged(qd[t], kd[t], vd[t], Kp, Vp, table, pos, 0, w.scale,
                             workspace=ws)
            pos += 1
    ms_tp = timer.run(turn_paged, max(1, reps // 4), 1, WARM_MS)
    out["decode_paged"] = {"ms_per_step": ms_tp / w.steps, "page_size": ps,
                           "gbs": b_dec / ms_tp / 1e6,
                           "frac_peak_hbm": b_dec / ms_tp / 1e6 / PEAK_HBM_GBS,
                           "vs_dense": ms_turn / ms_tp}

    # verification of drafted tokens (speculative decoding): the first
    # n_draft decode inputs of every dialogue as one causal answer chunk
    # through the paged cache, against n_draft decode steps
    n_draft = 8
    cu_d = torch.arange(B + 1, dtype=torch.int32, device="cuda") * n_draft

    def chunk(x):
        return x[:n_draft].transpose(0, 1).reshape(B * n_draft, *x.shape[2:]).contiguous()
    qv, kv, vv = chunk(qd), chunk(kd), chunk(vd)
    ms_ver = timer.run(lambda: ops.prefill_paged(qv, kv, vv, Kp, Vp, table, pos0, cu_d,
                                                 n_draft, False, w.scale), reps, warmup,
                       WARM_MS)
    out["verify_paged"] = {"drafts": n_draft, "ms": ms_ver,
                           "decode_steps_ms": n_draft * ms_tp / w.steps,
                           "speedup_vs_decode": n_draft * ms_tp / w.steps / ms_ver}

    # ChatGLM-style 2-D positions (the new query is the dialogue's segment
    # 2 x 16 = 32, offsets 0..L-1): the prefill with the rotation fused into
    # the append and the query load, against rotating q and k first
    p1 = torch.full((qn.shape[0],), 32, dtype=torch.int32, device="cuda")
    p2 = torch.cat([torch.arange(int(n), dtype=torch.int32) for n in w.new_lens]).cuda()
    ms_rf = timer.run(lambda: ops.prefill_cached_rope2d(qn, kn, vn, Kc, Vc, lens, cu, mx,
                                                        p1, p2, True, scale=w.scale),
                      reps, warmup, WARM_MS)
    qr, kr = qn.clone(), kn.clone()

    def unfused():
        ops.rope2d_(qr, p1, p2)
        ops.rope2d_(kr, p1, p2)
        ops.prefill_cached_segment(qr, kr, vn, Kc, Vc, lens, cu, mx, True, w.scale)
    ms_ru = timer.run(unfused, reps, warmup, WARM_MS)
    ms_rq = timer.run(lambda: ops.rope2d_(qr, p1, p2), reps, warmup, WARM_MS)
    rq_bytes = 2 * qr.numel() * 2  # bf16 read + write
    out["prefill_rope2d"] = {"fused_ms": ms_rf, "unfused_ms": ms_ru, "plain_ms": ms_pf,
                             "rope_q_ms": ms_rq, "rope_q_gbs": rq_bytes / ms_rq / 1e6,
                             "rope_q_frac_peak_hbm": rq_bytes / ms_rq / 1e6 / PEAK_HBM_GBS}
    return out


def read_ceiling(timer, nbytes=4 << 30):
    """Streaming-read rate of a plain kernel (libism_calib.so): the practical
    ceiling for the HBM-bound decode, reported beside the 8 TB/s spec.
    Best of a few grid sizes over a 4 GiB buffer."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2408_00539_amd", "libism_calib.so")
    fn = ctypes.CDLL(path).ism_calib_stream_read
    fn.restype = ctypes.c_int64
    fn.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                   ctypes.c_void_p]
    buf = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    by_grid = {}
    for grid in (1024, 2048, 4096, 8192):
        def run():
            n = fn(buf.data_ptr(), nbytes, out.data_ptr(), grid, stream)
            if n < 0:
                raise RuntimeError("stream-read launch failed")
            return n
        n = run()
        ms = timer.run(run, 10, 2, WARM_MS / 4)
        by_grid[grid] = n / ms / 1e6
    best = max(by_grid.values())
    del buf
    return {"bytes": n, "gbs": best, "frac_peak_hbm": best / PEAK_HBM_GBS,
            "gbs_by_grid": {str(g): round(v, 1) for g, v in by_grid.items()}}


def bench_expansion(w, timer, reps, warmup, ism_step_ms):
    """Training on the dialogues of ``w`` the way a prefix-mask model must
    (Sec. 1): every dialogue expanded into one sample per turn (history up to
    Q_k as a bidirectional prefix, then A_k), one forward + backward over the
    expanded batch; against ISM's single pass over the same dialogues."""
    from paper_2408_00539_amd import ops, workloads as W
    import torch
    exp, src = W.prefix_expansion(w.segs)
    segs = ops.Segments.from_host(exp.cu_seqlens, exp.cu_segs, exp.seg_is_query)
    ix = torch.from_numpy(src).cuda()
    q = dev(w.q).index_select(0, ix)
    k = dev(w.k).index_select(0, ix)
    v = dev(w.v).index_select(0, ix)
    do = dev(w.do).index_select(0, ix)
    pairs = visible_pairs(exp)
    flop = 14 * w.d * w.hq * pairs

    def step():
        o, lse = ops.fwd(q, k, v, segs, w.scale)
        ops.bwd(q, k, v, o, lse, do, segs, w.scale)
    ms = timer.run(step, reps, warmup, WARM_MS)
    return {"train_prefix_expansion": {
        "workload": "the dialogues of the training step, one sample per turn",
        "samples": exp.batch, "tokens": exp.total, "ms": ms,
        "tflops": flop / ms / 1e9, "flop": flop,
        "ism_step_ms": ism_step_ms, "ism_speedup": ms / ism_step_ms}}


LAT_B, LAT_TURNS, LAT_Q, LAT_A = 40, 20, 40, 160   # Sec. 3.6 latency workload
LAT_HQ, LAT_HKV, LAT_D = 32, 8, 128


def bench_latency(timer, reps=5, seed=5):
    """The paper's latency experiment (Sec. 3.6: forty simulated dialogues of
    20 turns, 40 query + 160 answer tokens per turn, context up to 4000) at
    the level of one attention layer with 32 query / 8 KV heads, head_dim 128,
    all forty dialogues batched. Per turn: time to first token = the new
    query's prefill under ISM (query segment through the reused cache),
    under the causal mask (the same rows causal) and under the prefix mask
    (which cannot reuse the cache: the whole prefix is recomputed as one
    bidirectional segment); time per output token = one decode step (the
    same operation under all three masks: an answer token sees everything
    before it). Inputs: seeded N(0, 1) bf16 drawn on the device."""
    from paper_2408_00539_amd import ops
    import torch
    B, T_ctx = LAT_B, LAT_TURNS * (LAT_Q + LAT_A)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def rnd(*shape):
        return torch.randn(*shape, generator=g, device="cuda",
                           dtype=torch.float32).to(torch.bfloat16)
    Q = rnd(B, T_ctx, LAT_HQ, LAT_D)
    K = rnd(B, T_ctx, LAT_HKV, LAT_D)
    V = rnd(B, T_ctx, LAT_HKV, LAT_D)
    kc = torch.zeros(B, LAT_HKV, T_ctx, LAT_D, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    cu_new = torch.arange(B + 1, dtype=torch.int32, device="cuda") * LAT_Q
    ws = torch.empty(ops.workspace_size(ops.ISM_OP_DECODE, B, 0, T_ctx, LAT_HQ,
                                        LAT_HKV, LAT_D, 0),
                     dtype=torch.uint8, device="cuda")
    scale = 1.0 / math.sqrt(LAT_D)
    out = {m: [] for m in ("ttft_ism_ms", "ttft_causal_ms", "ttft_prefix_ms",
                           "tpot_ms")}
    for n in range(LAT_TURNS):
        C = n * (LAT_Q + LAT_A)
        P = C + LAT_Q
        qn = Q[:, C:P].reshape(B * LAT_Q, LAT_HQ, LAT_D).contiguous()
        kn = K[:, C:P].reshape(B * LAT_Q, LAT_HKV, LAT_D).contiguous()
        vn = V[:, C:P].reshape(B * LAT_Q, LAT_HKV, LAT_D).contiguous()
        clen = torch.full((B,), C, dtype=torch.int32, device="cuda")
        for mode, isq in (("ttft_ism_ms", True), ("ttft_causal_ms", False)):
            out[mode].append(timer.run(lambda: ops.prefill_cached_segment(
                qn, kn, vn, kc, vc, clen, cu_new, LAT_Q, isq, scale), reps, 2,
                LAT_WARM_MS))
        # prefix mask: the whole prefix, one bidirectional segment per dialogue
        cu = np.arange(B + 1, dtype=np.int32) * P
        psegs = ops.Segments.from_host(cu, cu, np.ones(B, np.uint8))
        qp = Q[:, :P].reshape(B * P, LAT_HQ, LAT_D).contiguous()
        kp = K[:, :P].reshape(B * P, LAT_HKV, LAT_D).contiguous()
        vp = V[:, :P].reshape(B * P, LAT_HKV, LAT_D).contiguous()
        out["ttft_prefix_ms"].append(timer.run(
            lambda: ops.fwd(qp, kp, vp, psegs, scale), reps, 2, LAT_WARM_MS))
        del qp, kp, vp
        # the answer, one token per step
        qd = Q[:, P:C + LAT_Q + LAT_A].transpose(0, 1).contiguous()
        kd = K[:, P:C + LAT_Q + LAT_A].transpose(0, 1).contiguous()
        vd = V[:, P:C + LAT_Q + LAT_A].transpose(0, 1).contiguous()
        pos = (P + torch.arange(LAT_A, dtype=torch.int32, device="cuda"))[:, None]
        pos = pos.expand(LAT_A, B).contiguous()

        def answer():
            for t in range(LAT_A):
                ops.decode(qd[t], kd[t], vd[t], kc, vc, pos[t], T_ctx, scale,
                           workspace=ws)
        # (a repeated answer writes the same keys to the same positions)
        out["tpot_ms"].append(timer.run(answer, 1, 1, LAT_WARM_MS) / LAT_A)
    res = {"workload": f"{B} dialogues x {LAT_TURNS} turns x ({LAT_Q} query + "
                       f"{LAT_A} answer) tokens, {LAT_HQ}/{LAT_HKV} heads, "
                       f"head_dim {LAT_D}, one attention layer",
           "turns_reported": [1, 5, 10, 15, 20]}
    for m, vals in out.items():
        res[m] = [round(vals[i - 1], 4) for i in res["turns_reported"]]
        res[m.replace("_ms", "_mean_ms")] = round(float(np.mean(vals)), 4)
    res["ttft_ism_minus_causal_us"] = round(
        1000 * (res["ttft_ism_mean_ms"] - res["ttft_causal_mean_ms"]), 2)
    return {"latency": res}


DG_B, DG_POS, DG_CAP, DG_HKV, DG_D = 32, 8192, 9216, 8, 128
DG_HQ = (8, 32, 48, 64)  # query heads per KV head: 1, 4, 6, 8


def bench_decode_groups(timer, reps=50, seed=6):
    """The decode step with grouped KV heads: 32 dialogues at position 8192
    (cache capacity 9216), 8 KV heads of 128, and 8, 32, 48 or 64 query
    heads (1, 4, 6 or 8 per KV head). Bytes per step: K and V of every key
    once, whatever the grouping (a workgroup serves all query heads of its
    KV head, up to 8). Inputs: seeded N(0, 1) bf16 drawn on the device."""
    from paper_2408_00539_amd import ops
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def rnd(*shape):
        return torch.randn(*shape, generator=g, device="cuda",
                           dtype=torch.float32).to(torch.bfloat16)
    kc, vc = rnd(DG_B, DG_HKV, DG_CAP, DG_D), rnd(DG_B, DG_HKV, DG_CAP, DG_D)
    kn, vn = rnd(DG_B, DG_HKV, DG_D), rnd(DG_B, DG_HKV, DG_D)
    lens = torch.full((DG_B,), DG_POS, dtype=torch.int32, device="cuda")
    nbytes = DG_B * DG_HKV * 2 * (DG_POS + 1) * DG_D * 2
    res = {"workload": f"{DG_B} dialogues at position {DG_POS}, {DG_HKV} KV heads, "
                       f"head_dim {DG_D}", "bytes_per_step": nbytes}
    for hq in DG_HQ:
        q = rnd(DG_B, hq, DG_D)
        # (a repeated step writes the same key to the same position)
        ms = timer.run(lambda: ops.decode(q, kn, vn, kc, vc, lens), reps, 5, WARM_MS)
        res[f"g{hq // DG_HKV}"] = {"hq": hq, "ms_per_step": round(ms, 4),
                                   "gbs": round(nbytes / ms / 1e6, 1),
                                   "frac_peak_hbm": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 4)}
    del kc, vc
    return {"decode_head_groups": res}


def _f64(bits):
    from paper_2408_00539_amd.workloads import bf16_bits_to_f32
    return bf16_bits_to_f32(bits).astype(np.float64)


def cpu_baseline(w4, w1=None, w2=None, w3=None, gpu4=None):
    """The fp64 oracle (test infrastructure, as it stands) on bounded samples
    of the workloads, on the host cores; one (dialogue, head) pair per
    thread, one BLAS thread each.

    Headline: the training step of workload 4 (oracle forward + backward)
    on the first `workers` (dialogue, head) pairs, in useful TFLOP/s.
    Beside it: the forward of workload 1 (all pairs) and of workload 2
    (`workers` pairs), and workload 3's cache path for one dialogue (the
    one-shot reference rows of its new query segment and 16 answer tokens,
    then the same 16 tokens as stepwise decode steps after the cached
    prefill, as the per-step time and its K/V bytes per second).

    gpu4 = (o, lse, dq, dk, dv), the device outputs of one step of workload
    4: after the timing, the headline sample's oracle results are compared
    with them on its pairs (max / mean absolute error per tensor, the
    parity bar's two terms), so the line carries the parity of what it
    timed."""
    import oracle
    from threadpoolctl import threadpool_limits
    cores = len(os.sched_getaffinity(0))
    workers = max(1, min(cores, 16))
    out = {"unit": "TFLOP/s", "cores": workers, "kind": "oracle",
           "cpu": _cpu_model(), "blas": _blas_name(), "legs": {}}

    def pairs_flop(w, pairs, per_pair):
        return per_pair * w.d * sum(_pairs_of_dialogue(w.segs, b) for b, _ in pairs)

    with threadpool_limits(limits=1):
        q, k, v, do = _f64(w4.q), _f64(w4.k), _f64(w4.v), _f64(w4.do)
        args = (w4.segs.cu_seqlens, w4.segs.cu_segs, w4.segs.seg_is_query, w4.scale)
        pairs = [(b, h) for b in range(w4.segs.batch) for h in range(w4.hq)][:workers]
        t0 = time.perf_counter()
        ref = oracle.fwd(q, k, v, *args, pairs=pairs, workers=workers)
        ref += oracle.bwd(q, k, v, do, *args, pairs=pairs, workers=workers)
        dt = time.perf_counter() - t0
        flop = pairs_flop(w4, pairs, 14)
        if gpu4 is not None:
            out["parity"] = _sample_parity(w4, pairs, gpu4, ref)
        out.update({"value": flop / dt / 1e12, "seconds": round(dt, 2),
                    "sample": f"fp64 oracle forward + backward of workload 4 (4 x 8192, "
                              f"32 heads, d 128) on {len(pairs)} of "
                              f"{w4.segs.batch * w4.hq} (dialogue, head) pairs, "
                              f"{workers} threads, {dt:.1f} s wall; useful FLOPs "
                              f"of those pairs (14 d per visible pair)"})
        del q, k, v, do
        from paper_2408_00539_amd import workloads as W
        w0 = W.make_workload(0)
        for name, w, full in (("fwd_small", w0, True), ("fwd_8x4096", w1, True),
                              ("fwd_gqa_2x16384", w2, False)):
            if w is None:
                continue
            q, k, v = _f64(w.q), _f64(w.k), _f64(w.v)
            args = (w.segs.cu_seqlens, w.segs.cu_segs, w.segs.seg_is_query, w.scale)
            pairs = [(b, h) for b in range(w.segs.batch) for h in range(w.hq)]
            if not full:
                pairs = pairs[:workers]
            t0 = time.perf_counter()
            oracle.fwd(q, k, v, *args, pairs=pairs, workers=workers)
            dt = time.perf_counter() - t0
            out["legs"][name] = {"value": pairs_flop(w, pairs, 4) / dt / 1e12,
                                 "unit": "TFLOP/s", "seconds": round(dt, 2),
                                 "pairs": len(pairs),
                                 "of_pairs": w.segs.batch * w.hq}
            del q, k, v
        if w3 is not None:
            out["legs"]["cache_32x8192"] = _cpu_cache_leg(oracle, w3, workers)
    return out


def _sample_parity(w, pairs, gpu, ref):
    """Max and mean absolute error of the device outputs against the
    oracle's on the (dialogue, head) pairs it computed."""
    names = ("O", "LSE", "dQ", "dK", "dV")
    cu = w.segs.cu_seqlens
    G = w.hq // w.hkv
    res = {"pairs": len(pairs)}
    for name, g, r in zip(names, gpu, ref):
        errs = []
        for b, h in pairs:
            s, e = int(cu[b]), int(cu[b + 1])
            hh = h // G if name in ("dK", "dV") else h
            if name == "LSE":
                gv, rv = g[hh, s:e], r[hh, s:e]
            else:
                gv, rv = g[s:e, hh], r[s:e, hh]
            errs.append(np.abs(gv.float().cpu().numpy().astype(np.float64) - rv).ravel())
        err = np.concatenate(errs)
        res[name] = {"max_abs": float(err.max()), "mean_abs": float(err.mean())}
    return res


def _cpu_cache_leg(oracle, w, workers, steps=16):
    """One dialogue of workload 3: the one-shot oracle forward of its new
    query segment and `steps` answer tokens over [history; Q_n; A_n] (the
    reference rows of the parity tests), and the stepwise path: cached
    prefill, then `steps` decode steps, each appending its key / value."""
    from concurrent.futures import ThreadPoolExecutor
    from paper_2408_00539_amd import workloads as W
    b, C, L = 0, w.hist_len, int(w.new_lens[0])
    r0, r1 = int(w.cu_new[0]), int(w.cu_new[1])
    kh = _f64(w.k_cache[0, :, :C]).transpose(1, 0, 2)
    vh = _f64(w.v_cache[0, :, :C]).transpose(1, 0, 2)
    qn, kn, vn = _f64(w.q_new[r0:r1]), _f64(w.k_new[r0:r1]), _f64(w.v_new[r0:r1])
    qd, kd, vd = (_f64(x[:steps, b]) for x in (w.q_dec, w.k_dec, w.v_dec))
    dia = W.segments_from_lengths([
        [(int(n), bool(f)) for n, f in zip(np.diff(w.hist.cu_segs[:33]),
                                            w.hist.seg_is_query[:32])]
        + [(L, True), (steps, False)]])
    n = C + L + steps
    qq = np.zeros((n, w.hq, w.d))
    qq[C:C + L], qq[C + L:] = qn, qd
    kk = np.concatenate([kh, kn, kd])
    vv = np.concatenate([vh, vn, vd])
    t0 = time.perf_counter()
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda h: oracle.fwd_rows(qq, kk, vv, dia.cu_seqlens, dia.cu_segs,
                                              dia.seg_is_query, w.scale, 0, h,
                                              rows=(C, n)), range(w.hq)))
    t_one = time.perf_counter() - t0
    t0 = time.perf_counter()
    _, _, kc, vc = oracle.prefill_cached(kh, vh, qn, kn, vn, w.scale)
    t_pf = time.perf_counter() - t0
    t0 = time.perf_counter()
    for t in range(steps):
        _, _, kc, vc = oracle.decode_step(kc, vc, qd[t], kd[t], vd[t], w.scale)
    t_dec = (time.perf_counter() - t0) / steps
    kv_bytes = 2 * w.hkv * w.d * 2 * (C + L + steps / 2 + 0.5)  # bf16 K+V per step
    return {"dialogues": 1, "of_dialogues": len(w.new_lens), "decode_steps": steps,
            "one_shot_rows_s": round(t_one, 3), "prefill_s": round(t_pf, 3),
            "decode_ms_per_step": round(1e3 * t_dec, 2),
            "decode_equiv_gbs": kv_bytes / t_dec / 1e9,
            "note": "one-shot rows use a thread per head; the stepwise path runs "
                    "on one thread"}


def _pairs_of_dialogue(segs, b):
    from types import SimpleNamespace
    cu = segs.cu_seqlens
    s, e = int(cu[b]), int(cu[b + 1])
    cs = np.asarray(segs.cu_segs)
    g0, g1 = int(np.searchsorted(cs, s)), int(np.searchsorted(cs, e))
    return visible_pairs(SimpleNamespace(
        cu_seqlens=np.array([0, e - s]), cu_segs=cs[g0:g1 + 1] - s,
        seg_is_query=np.asarray(segs.seg_is_query)[g0:g1]))


def _blas_name():
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        return f"{b.get('name')} {b.get('version')}"
    except Exception:  # older numpy: no dict form
        return None


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def kernel_source_hash():
    """sha256 over the library's kernel sources (names and contents)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2408_00539_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def recorded_traffic():
    """HBM bytes per backward launch from the committed counter record, or
    None when there is none or the kernels changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec.get("bwd_bytes_per_launch")


def _counter_means(path, counter):
    """Mean per dispatch of one counter, per kernel, from a rocprofv3
    counter_collection.csv (kernel name -> (mean KiB, dispatches))."""
    import csv
    sums, counts = {}, {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            k = _short_kernel(r["Kernel_Name"])
            sums[k] = sums.get(k, 0.0) + float(r["Counter_Value"])
            counts[k] = counts.get(k, 0) + 1
    return {k: (sums[k] / counts[k], counts[k]) for k in sums}


def _short_kernel(name):
    import re
    if name.startswith("_ZN3ism12_GLOBAL__N_1"):
        rest = name[len("_ZN3ism12_GLOBAL__N_1"):]
        m = re.match(r"(\d+)", rest)
        n = int(m.group(1))
        base = rest[len(m.group(1)):len(m.group(1)) + n]
        t = re.match(r"ILi(\d+)E", rest[len(m.group(1)) + n:])
        return base + (f"<{t.group(1)}>" if t else "")
    name = name.replace("void ", "").replace("ism::(anonymous namespace)::", "")
    name = name.replace("(anonymous namespace)::", "")
    return name.replace("ism::", "").split("(")[0]


def write_traffic_record(fetch_copy, fetch_step, write_copy, write_step,
                         fetch_cache=None, write_cache=None):
    """Turn the counter passes into the traffic record bench.py reports:
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of each kernel, scaled by
    what the same counters read for the plain COPY_BYTES copy."""
    fc = _counter_means(fetch_copy, "FETCH_SIZE")
    wc = _counter_means(write_copy, "WRITE_SIZE")
    copy_f = max(v for v, _ in fc.values())
    copy_w = max(v for v, _ in wc.values())
    sf = COPY_BYTES / 1024 / copy_f
    sw = COPY_BYTES / 1024 / copy_w
    rec = {"kernel_source_sha256": kernel_source_hash(),
           "workload": "training step, 4 dialogues x 8192 tokens, 32 heads, "
                       "head_dim 128 (cache path: 32 x 8192, 32 heads)",
           "copy_calibration": {"copy_bytes": COPY_BYTES,
                                "FETCH_SIZE_KiB": round(copy_f, 1),
                                "WRITE_SIZE_KiB": round(copy_w, 1),
                                "scale_fetch": round(sf, 4),
                                "scale_write": round(sw, 4)},
           "kernels": {}}
    passes = [(fetch_step, write_step)]
    if fetch_cache and write_cache:
        passes.append((fetch_cache, write_cache))
    for fp, wp in passes:
        fk, wk = _counter_means(fp, "FETCH_SIZE"), _counter_means(wp, "WRITE_SIZE")
        for k in fk:
            if k not in wk or "elementwise" in k or "copyBuffer" in k:
                continue
            f, w = fk[k][0], wk[k][0]
            rec["kernels"][k] = {"FETCH_SIZE_KiB": round(f, 1),
                                 "WRITE_SIZE_KiB": round(w, 1),
                                 "bytes": int(sf * f * 1024 + sw * w * 1024)}
    kb = rec["kernels"]
    rec["bwd_bytes_per_launch"] = sum(
        kb[k]["bytes"] for k in kb if k.startswith(("bwd_prep_kernel", "dkv_kernel", "dq_kernel")))
    rec["fwd_bytes_per_launch"] = sum(
        kb[k]["bytes"] for k in kb if k.startswith("fwd_kernel<128, false"))
    dec = [k for k in kb if k.startswith("decode_split_kernel")]
    if dec:
        # the dense cache's kernels (the paged ones carry PAGED = true)
        rec["decode_bytes_per_step"] = sum(
            kb[k]["bytes"] for k in kb
            if k.startswith("decode_combine")
            or (k.startswith("decode_split") and "true" not in k))
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    lines = ["| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes (scaled) |",
             "|---|---|---|---|"]
    for k, v in kb.items():
        lines.append(f"| {k} | {v['FETCH_SIZE_KiB']:.0f} | {v['WRITE_SIZE_KiB']:.0f} | "
                     f"{v['bytes'] / 1e9:.3f} GB |")
    print("\n".join(lines))
    print(f"scale: fetch {sf:.3f}, write {sw:.3f}; backward {rec['bwd_bytes_per_launch'] / 1e9:.3f} GB"
          f" per launch; sha256 {rec['kernel_source_sha256']}")


def recorded_decode_traffic():
    """HBM bytes per decode step from the counter record (or None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec.get("decode_bytes_per_step")


def calibrate_copy():
    """A plain device copy of COPY_BYTES, ten times (for the counter scale)."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "copies": 10}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=["all", "step", "gqa", "bwd", "cache",
                                       "expansion", "latency", "decode_groups"],
                    default="all")
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--write-traffic-record", nargs="+", metavar="CSV",
                    help="counter_collection.csv files: FETCH_SIZE of the "
                    "copy, of the step, WRITE_SIZE of the copy, of the step "
                    "[, FETCH_SIZE and WRITE_SIZE of the cache path]; writes "
                    "the traffic record (no GPU needed)")
    args = ap.parse_args()
    if args.write_traffic_record:
        write_traffic_record(*args.write_traffic_record)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this library has no multi-GPU "
              "path (see the sharding design); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2408_00539_amd import ops, workloads as W
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    ops.lib()
    if args.calibrate_copy:
        calibrate_copy()
        return
    timer = Timer()
    if args.only in ("gqa", "bwd", "cache", "expansion", "latency", "decode_groups"):
        paths = {}
        if args.only == "gqa":
            w2 = W.make_workload(2)
            t2 = bench_training(w2, timer, 10, 2, False)
            paths["fwd_gqa"] = dict(t2["fwd"], workload="2x16384 h32/kv8 d128")
        elif args.only == "bwd":
            w4 = W.make_workload(4)
            t4 = bench_training(w4, timer, 5, 1, True)
            paths["bwd"] = dict(t4["bwd"], workload="4x8192 h32 d128")
        elif args.only == "cache":
            paths.update(bench_cache(W.make_workload(3), timer, 8, 2))
        elif args.only == "expansion":
            w1 = W.make_workload(1)
            w1.do = W.packed_tensor(w1.seed, W.DO, w1.segs.cu_seqlens, w1.hq, w1.d)
            tr = bench_training(w1, timer, 5, 1, True)
            paths.update(bench_expansion(w1, timer, 3, 1, tr["step"]["ms"]))
        elif args.only == "decode_groups":
            paths.update(bench_decode_groups(timer))
        else:
            paths.update(bench_latency(timer))
        print(json.dumps({"paths": paths}), flush=True)
        return

    # the headline: the training step of workload 4
    log("generating workload 4 ...")
    w4 = W.make_workload(4)
    torch.cuda.synchronize()
    tr = bench_training(w4, timer, args.steps, args.warmup, True)
    step_ms, step_flop = tr["step"]["ms"], tr["step"]["flop"]
    log(f"step: {step_ms:.3f} ms, {step_flop / step_ms / 1e9:.1f} TFLOP/s")
    paths = {"fwd_4x8192": dict(tr["fwd"], workload="4x8192 h32 d128"),
             "bwd": dict(tr["bwd"], workload="4x8192 h32 d128")}
    dom = tr["bwd"]
    w1 = w2 = w3 = None
    if args.only == "all":
        log("generating workload 1 ...")
        w1 = W.make_workload(1)
        w1.do = W.packed_tensor(w1.seed, W.DO, w1.segs.cu_seqlens, w1.hq, w1.d)
        t1 = bench_training(w1, timer, 10, 2, True)
        paths["fwd"] = dict(t1["fwd"], workload="8x4096 h32 d128")
        paths["step_8x4096"] = dict(t1["step"], workload="8x4096 h32 d128 (prep+fwd+bwd)")
        paths["bwd_8x4096"] = dict(t1["bwd"], workload="8x4096 h32 d128")
        log("generating workload 2 ...")
        w2 = W.make_workload(2)
        t2 = bench_training(w2, timer, 10, 2, False)
        paths["fwd_gqa"] = dict(t2["fwd"], workload="2x16384 h32/kv8 d128")
        log("generating workload 3 ...")
        w3 = W.make_workload(3)
        paths.update(bench_cache(w3, timer, 8, 2))
        torch.cuda.empty_cache()
        log("prefix-mask expansion of workload 1's dialogues ...")
        paths.update(bench_expansion(w1, timer, 3, 1, t1["step"]["ms"]))
        torch.cuda.empty_cache()
        log("latency turns ...")
        paths.update(bench_latency(timer))
        torch.cuda.empty_cache()
        log("decode with grouped KV heads ...")
        paths.update(bench_decode_groups(timer))
        torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        # one more step of workload 4, its outputs for the parity report
        segs4 = ops.Segments.from_host(w4.segs.cu_seqlens, w4.segs.cu_segs,
                                       w4.segs.seg_is_query)
        q4, k4, v4, do4 = dev(w4.q), dev(w4.k), dev(w4.v), dev(w4.do)
        o4, l4 = ops.fwd(q4, k4, v4, segs4, w4.scale)
        gpu4 = (o4, l4) + tuple(ops.bwd(q4, k4, v4, o4, l4, do4, segs4, w4.scale))
        torch.cuda.synchronize()
        log("timing the CPU oracle ...")
        cpu = cpu_baseline(w4, w1, w2, w3, gpu4)

    value = step_flop / step_ms / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "tokens_per_s": round(tr["step"]["tokens_per_s"], 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "ISM training step (prep + forward with LSE + backward), "
                   "4 dialogues x 8192 tokens, 16 turns, 32 heads, head_dim 128",
                   "global_batch": 4, "seq_len": 8192, "heads": 32,
                   "head_dim": 128, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma",
                     "kernel": "ism_attn_bwd on the step's inputs (all its launches)",
                     "achieved": round(dom["tflops"], 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(dom["tflops"] / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic()},
        "cpu_baseline": cpu,
        "device": device_info(),
        "paths": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv)
                      for kk, vv in v.items()} for k, v in paths.items()},
    }
    print(json.dumps(line), flush=True)

if __name__ == "__main__":
    main()
