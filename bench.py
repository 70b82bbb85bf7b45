"""Benchmark of the SpecFLASH draft-verify hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step is one pass of the whole hot path over one batch of synthetic
input with every tensor already resident in HBM:
    sd_latent_compress (Eq. 3) -> sd_semi_ar_layer (the draft's step for one
    accepted token and the k placeholders of each sequence) ->
    sd_verify_attention -> sd_lm_head_probs (the k+1 target rows) ->
    sd_spec_accept -> sd_spec_accept_logits
(the draft side, then the target side, as in a drafting round)
Default workload: "long-video" (batch 4, GQA 64/8 heads, head dim 128, KV
length 65536, block k = 8; compression of 16384 tokens of width 8192 to 512
latents over 64 heads; an LM head of width 8192 over a 152064-token
vocabulary for the 36 target rows; sampled acceptance over that vocabulary
at temperature 0.7).  The acceptance consumes synthetic p and q with
realistic acceptance rates, not the head's output (its weights are random);
the acceptance from logits runs on the logits of the same draws (temperature
softmax and Philox uniforms on the device).  The draft layer has the
target's width and heads (8192, 64 / 8) with a SwiGLU MLP of width 28672,
over a cached context of 544 + 3 b positions.

Prints one JSON line.  `value` is the verify step's KV-read rate: bytes of
K and V the step must read once, divided by the time of verification
attention plus acceptance, in TB/s.  Per-kernel times come from HIP events
on the stream the kernels run on.  `roofline` describes the dominant kernel
(the longest per step); `rooflines` lists all six.  `traffic` is the HBM
bytes per launch measured with rocprofv3 counters (profiles/), or null when
the kernel's sources changed since they were taken.  `cpu_baseline` times
the plain CPU oracle on a bounded sample of the same workload and scales it
to the whole step.
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("verify-step µs & KV-read HBM TB/s at long KV; "
          "latent-compress MFMA TFLOP/s")
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 / fp16 matrix cores
FP32_VALU_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long-video")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the CPU oracle")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip timing the other workloads' compression, verification and acceptance")
    ap.add_argument("--workload-steps", type=int, default=30,
                    help="timed calls per operation for each of the other workloads")
    ap.add_argument("--core-only", action="store_true",
                    help="time only the workload's compression, verification and acceptance "
                         "(one JSON line of per-operation statistics; for profiling runs)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (for counter scaling)")
    return ap.parse_args()


def to_dev(t, dev):
    import numpy as np
    import torch
    if t.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(t.bits).view(np.int16)).view(
            torch.bfloat16).to(dev)
    return torch.from_numpy(np.ascontiguousarray(t.values)).to(dev)


def accept_bytes(p, n):
    """Algorithmic bytes of one acceptance call: the k test scalars plus one
    full vocabulary pass over the row that is sampled (p_n and q_n when a
    draft was rejected, p_k alone when all were accepted)."""
    B, kp1, V = p.shape
    k = kp1 - 1
    total = 0
    for nb in n:
        total += (2 * V if nb < k else V) * 4 + k * 4 * 3
    return total


def accept_logits_bytes(w, n):
    """Algorithmic bytes of one acceptance from float32 logits: every target
    and draft row once (the softmax statistics), then the sampled row pass
    over p_n and q_n (p_k alone after full acceptance)."""
    k, V = w.block, w.vocab
    total = 0
    for nb in n:
        total += (2 * k + 1) * V * 4 + (2 * V if nb < k else V) * 4
    return total


def op_stats(ms):
    """Per-call times (ms) -> median, p10, p90 and mean in microseconds."""
    import numpy as np
    us = np.asarray(ms, dtype=np.float64) * 1e3
    return {"median_us": float(np.median(us)), "p10_us": float(np.percentile(us, 10)),
            "p90_us": float(np.percentile(us, 90)), "mean_us": float(us.mean()), "calls": int(us.size)}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


# Targets on the roofline fraction of the gated operations, per workload:
# verification attention >= 70% of HBM peak on the long-KV workloads and
# latent compression >= 50% of the bf16 matrix-core peak where it is
# matrix-core bound.
GATES = {("batched-paged", "verify_attention"): 0.70, ("long-video", "verify_attention"): 0.70,
         ("qwen2vl-7b-video", "latent_compress"): 0.50, ("long-video", "latent_compress"): 0.50}


def time_workload_ops(w, dev, steps, warmup):
    """Compression, verification attention and acceptance of one workload,
    timed in pipeline order (the three operations of the metric) with HIP
    events on the stream they run on; inputs resident in HBM.  Returns the
    per-operation statistics with rates and roofline fractions."""
    import numpy as np
    import torch

    import paper_2505_12728_amd as sd
    from paper_2505_12728_amd import synth

    mode = "sampled" if "sampled" in w.modes else "greedy"
    comp = synth.compress_inputs(w)
    ver = synth.verify_inputs(w)
    acc = synth.accept_inputs(w, mode)
    lat_d, feats_d = to_dev(comp[0], dev), to_dev(comp[1], dev)
    q_d, k_d, v_d = to_dev(ver["q"], dev), to_dev(ver["k_cache"], dev), to_dev(ver["v_cache"], dev)
    kl_d = torch.from_numpy(ver["kv_len"]).to(dev)
    pt_d = None if ver["page_table"] is None else torch.from_numpy(ver["page_table"]).to(dev)
    p_d, qq_d = torch.from_numpy(acc["p"]).to(dev), torch.from_numpy(acc["q"]).to(dev)
    dr_d, u_d = torch.from_numpy(acc["draft"]).to(dev), torch.from_numpy(acc["u"]).to(dev)
    dt_code = sd.SD_BF16 if w.dtype == "bf16" else sd.SD_F32
    amode = sd.SD_ACCEPT_SAMPLED if mode == "sampled" else sd.SD_ACCEPT_GREEDY
    c_out = torch.empty((w.c_batch, w.c_latents, w.c_width), dtype=torch.float32, device=dev)
    c_ws_n = sd.sd_latent_compress_workspace_size(w.c_batch, w.c_tokens, w.c_latents, w.c_width,
                                                  w.c_heads, dt_code)
    c_ws = torch.zeros(c_ws_n, dtype=torch.uint8, device=dev) if c_ws_n else None
    v_out = torch.empty((w.batch, w.block, w.hq, w.head_dim), dtype=torch.float32, device=dev)
    v_lse = torch.empty((w.batch, w.block, w.hq), dtype=torch.float32, device=dev)
    cap = w.kv_len if not w.paged else 16 * ver["max_pages"]
    v_ws = torch.zeros(sd.sd_verify_workspace_size(w.batch, w.block, w.hq, w.hkv, w.head_dim, cap,
                                                   dt_code), dtype=torch.uint8, device=dev)
    a_ws = torch.zeros(max(1, sd.sd_spec_accept_workspace_size(w.batch, w.block, w.vocab, amode)),
                       dtype=torch.uint8, device=dev)
    n_out = torch.empty((w.batch,), dtype=torch.int32, device=dev)
    t_out = torch.empty((w.batch, w.block + 1), dtype=torch.int32, device=dev)
    scale = 1.0 / math.sqrt(w.head_dim)

    def one(ev=None):
        if ev is not None:
            ev[0].record()
        sd.sd_latent_compress(lat_d, feats_d, w.c_heads, 1.0, out=c_out, workspace=c_ws)
        if ev is not None:
            ev[1].record()
        sd.sd_verify_attention(q_d, k_d, v_d, kl_d, scale=scale, page_table=pt_d, out=v_out,
                               lse=v_lse, workspace=v_ws)
        if ev is not None:
            ev[2].record()
        sd.sd_spec_accept(p_d, qq_d, dr_d, u_d, amode, n_accepted=n_out, tokens=t_out,
                          workspace=a_ws)
        if ev is not None:
            ev[3].record()

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for e in events:
        one(e)
    torch.cuda.synchronize()
    comp_ms = [e[0].elapsed_time(e[1]) for e in events]
    ver_ms = [e[1].elapsed_time(e[2]) for e in events]
    acc_ms = [e[2].elapsed_time(e[3]) for e in events]
    kv_bytes = synth.verify_kv_bytes(w, ver["kv_len"])
    flops = synth.compress_flops(w)
    a_bytes = accept_bytes(acc["p"], n_out.cpu().numpy())
    peak_c = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_VALU_PEAK_TFLOPS
    out = {"dtype": w.dtype, "accept_mode": mode}
    for name, ms, work, peak, unit in (
            ("latent_compress", comp_ms, flops, peak_c, "TFLOP/s"),
            ("verify_attention", ver_ms, kv_bytes, HBM_PEAK_GBS, "GB/s"),
            ("spec_accept", acc_ms, a_bytes, HBM_PEAK_GBS, "GB/s")):
        st = op_stats(ms)
        scale_ = 1e12 if unit == "TFLOP/s" else 1e9
        rate = work / (st["median_us"] * 1e-6) / scale_
        st.update({"algorithmic": work, "unit": unit, "achieved_at_median": rate, "peak": peak,
                   "frac_at_median": rate / peak,
                   "frac_at_p90": work / (st["p90_us"] * 1e-6) / scale_ / peak})
        gate = GATES.get((w.name, name))
        if gate is not None:
            st["target_frac"] = gate
            st["target_met_at_median"] = bool(st["frac_at_median"] >= gate)
        out[name] = st
    if w.dtype == "bf16":
        # the int8 draft's compressor on the same inputs quantised to int8
        # rows with power-of-two scales (same matrix-core work, half the
        # feature bytes)
        q = synth.compress_q8_inputs(w)
        qd = {k_: torch.from_numpy(v_).to(dev) for k_, v_ in q.items()}
        n8 = sd.sd_latent_compress_q8_workspace_size(w.c_batch, w.c_tokens, w.c_latents, w.c_width, w.c_heads)
        ws8 = torch.zeros(max(n8, 1), dtype=torch.uint8, device=dev)

        def q8():
            sd.sd_latent_compress_q8(qd["latents_q"], qd["latent_exp"], qd["feats_q"], qd["feat_exp"],
                                     w.c_heads, 1.0, out=c_out, workspace=ws8)

        for _ in range(warmup):
            q8()
        ev8 = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for e in ev8:
            e[0].record()
            q8()
            e[1].record()
        torch.cuda.synchronize()
        st = op_stats([e[0].elapsed_time(e[1]) for e in ev8])
        rate = flops / (st["median_us"] * 1e-6) / 1e12
        st.update({"algorithmic": flops, "unit": "TFLOP/s", "achieved_at_median": rate, "peak": BF16_PEAK_TFLOPS,
                   "frac_at_median": rate / BF16_PEAK_TFLOPS, "bytes": synth.compress_q8_bytes(w),
                   "outside_step": True})
        out["latent_compress_q8"] = st
        del qd, ws8
    vs = [a + b for a, b in zip(ver_ms, acc_ms)]
    out["verify_step"] = op_stats(vs)
    out["verify_step"]["kv_read_tbps_at_median"] = kv_bytes / (out["verify_step"]["median_us"] * 1e-6) / 1e12
    return out


def cpu_baseline(w, comp, ver, acc, mode, lm, accl, dr):
    """Time the oracle on a bounded sample and scale it to one whole step."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    lat, feats = comp
    dh = w.c_width // w.c_heads
    g = w.hq // w.hkv
    scale = 1.0 / math.sqrt(w.head_dim)
    # compression: up to 16 (sequence, head) pairs, every latent and token
    t0 = time.perf_counter()
    pairs_c = [(i % w.c_batch, (7 * i) % w.c_heads) for i in range(min(16, w.c_batch * w.c_heads))]
    for b, h in pairs_c:
        cols = slice(h * dh, (h + 1) * dh)
        oracle.latent_compress(lat.values[:, cols], feats.values[b:b + 1, :, cols], 1, 1.0)
    tc = (time.perf_counter() - t0) / len(pairs_c) * (w.c_batch * w.c_heads)
    # verification: up to 8 (sequence, KV head) pairs over the whole cache
    t0 = time.perf_counter()
    pairs_v = [(i % w.batch, (3 * i) % w.hkv) for i in range(min(8, w.batch * w.hkv))]
    for b, hk in pairs_v:
        q = ver["q"].values[b:b + 1, :, hk * g:(hk + 1) * g]
        if ver["page_table"] is None:
            oracle.verify_attention(q, ver["k_cache"].values[b:b + 1, :, hk:hk + 1],
                                    ver["v_cache"].values[b:b + 1, :, hk:hk + 1],
                                    ver["kv_len"][b:b + 1], scale)
        else:
            oracle.verify_attention(q, ver["k_cache"].values[:, hk:hk + 1],
                                    ver["v_cache"].values[:, hk:hk + 1], ver["kv_len"][b:b + 1],
                                    scale, page_table=ver["page_table"][b:b + 1])
    tv = (time.perf_counter() - t0) / len(pairs_v) * (w.batch * w.hkv)
    # acceptance: every sequence
    t0 = time.perf_counter()
    oracle.spec_accept(acc["p"], acc["q"], acc["draft"], acc["u"], mode)
    ta = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.spec_accept_logits(accl["target_logits"], accl["draft_logits"], accl["draft"],
                              accl["philox_seed"], accl["philox_offset"], accl["temperature"], mode)
    tal = time.perf_counter() - t0
    # LM head: one row over the whole vocabulary (logits 8192 entries at a time)
    R = lm["hidden"].shape[0]
    t0 = time.perf_counter()
    z = np.concatenate([oracle.lm_head_logits(lm["hidden"].values[:1], lm["weight"].values[v:v + 8192])
                        for v in range(0, w.vocab, 8192)], axis=1)
    oracle.softmax_temperature(z, lm["temperature"])
    tl = (time.perf_counter() - t0) * R
    # draft layer step: the first sequence's rows (the oracle's cost grows
    # with the rows), scaled to the batch
    Wd = {k: (v.values if hasattr(v, "values") else v) for k, v in dr["weights"].items()}
    t0 = time.perf_counter()
    oracle.semi_ar_layer(dr["u"].values[:1], Wd, dr["k_cache"].values[:1], dr["v_cache"].values[:1],
                         dr["pos"][:1], dr["hq"], dr["hkv"], dr["eps"], dr["theta"])
    td = (time.perf_counter() - t0) * dr["u"].shape[0]
    return {"compress_s": tc, "verify_s": tv, "accept_s": ta, "lm_head_s": tl, "accept_logits_s": tal,
            "draft_layer_s": td, "threads": threads, "cpu_model": cpu_model(),
            "sample": f"compress {len(pairs_c)} of {w.c_batch * w.c_heads} (sequence, head) "
                      f"pairs, verify {len(pairs_v)} of {w.batch * w.hkv} (sequence, KV head) "
                      f"pairs, acceptance (from p, q and from logits) of all {w.batch} sequences, "
                      f"LM head 1 of {R} rows, draft layer 1 of {dr['u'].shape[0]} sequences; "
                      f"scaled linearly"}


def counter_traffic(workload):
    """HBM bytes per launch from the committed counter summary of `workload`.

    profiles/<workload>_hbm_counters.md holds FETCH_SIZE / WRITE_SIZE per
    dispatch (calibrated against a plain device copy) together with the
    SHA-256 of the sources each kernel was built from.  A kernel whose
    sources have changed since gets None (its counters no longer apply).
    """
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_counters.md")
    if not os.path.exists(path):
        return {}
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return {}
    data = json.loads(text[start + 7:text.index("```", start + 7)])
    csrc = os.path.join(ROOT, "paper_2505_12728_amd", "csrc")
    out = {}
    for name, k in data["kernels"].items():
        digest = hashlib.sha256()
        for f in k["sources"]:
            with open(os.path.join(csrc, f), "rb") as fh:
                digest.update(fh.read())
        out[name] = k["hbm_bytes_per_launch"] if digest.hexdigest()[:16] == k["source_sha256_16"] else None
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the hot path is "
              "measured on one GPU's share; no multi-GPU run exists in this build.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2505_12728_amd as sd
    from paper_2505_12728_amd import synth

    sd.library()   # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.workload(args.workload)
    if args.core_only:
        if args.copy_calibration_mib:
            src = torch.empty(args.copy_calibration_mib << 20, dtype=torch.uint8, device=dev)
            torch.empty_like(src).copy_(src)
            torch.cuda.synchronize()
        print(f"[bench] core operations of {w.name}", file=sys.stderr, flush=True)
        ops_ = time_workload_ops(w, dev, args.steps, args.warmup)
        print(json.dumps({"workload": w.name, "steps": args.steps, "warmup": args.warmup, "ops": ops_}),
              flush=True)
        return
    mode = "sampled" if "sampled" in w.modes else "greedy"
    print(f"[bench] generating workload {w.name}", file=sys.stderr, flush=True)
    comp = synth.compress_inputs(w)
    ver = synth.verify_inputs(w)
    acc = synth.accept_inputs(w, mode)
    accl = synth.accept_logits_inputs(w, mode)
    lm = synth.lm_inputs(w)
    dr = synth.draft_inputs(w)

    lat_d, feats_d = to_dev(comp[0], dev), to_dev(comp[1], dev)
    q_d, k_d, v_d = to_dev(ver["q"], dev), to_dev(ver["k_cache"], dev), to_dev(ver["v_cache"], dev)
    kl_d = torch.from_numpy(ver["kv_len"]).to(dev)
    pt_d = None if ver["page_table"] is None else torch.from_numpy(ver["page_table"]).to(dev)
    p_d = torch.from_numpy(acc["p"]).to(dev)
    qq_d = torch.from_numpy(acc["q"]).to(dev)
    dr_d = torch.from_numpy(acc["draft"]).to(dev)
    u_d = torch.from_numpy(acc["u"]).to(dev)
    zt_d = torch.from_numpy(accl["target_logits"]).to(dev)
    zd_d = torch.from_numpy(accl["draft_logits"]).to(dev)
    drl_d = torch.from_numpy(accl["draft"]).to(dev)
    h_d, wt_d = to_dev(lm["hidden"], dev), to_dev(lm["weight"], dev)
    du_d = to_dev(dr["u"], dev)
    dw_d = {k: (to_dev(v, dev) if hasattr(v, "bits") else torch.from_numpy(v).to(dev))
            for k, v in dr["weights"].items()}
    dkc_d, dvc_d = to_dev(dr["k_cache"], dev), to_dev(dr["v_cache"], dev)
    dpos_d = torch.from_numpy(dr["pos"]).to(dev)
    dt_code = sd.SD_BF16 if w.dtype == "bf16" else sd.SD_F32
    amode = sd.SD_ACCEPT_SAMPLED if mode == "sampled" else sd.SD_ACCEPT_GREEDY

    # outputs and workspaces allocated once, outside the timed region
    c_out = torch.empty((w.c_batch, w.c_latents, w.c_width), dtype=torch.float32, device=dev)
    c_ws_n = sd.sd_latent_compress_workspace_size(w.c_batch, w.c_tokens, w.c_latents, w.c_width,
                                                  w.c_heads, dt_code)
    c_ws = torch.zeros(max(c_ws_n, 1), dtype=torch.uint8, device=dev) if c_ws_n else None
    v_out = torch.empty((w.batch, w.block, w.hq, w.head_dim), dtype=torch.float32, device=dev)
    v_lse = torch.empty((w.batch, w.block, w.hq), dtype=torch.float32, device=dev)
    cap = w.kv_len if not w.paged else 16 * ver["max_pages"]
    v_ws = torch.zeros(sd.sd_verify_workspace_size(w.batch, w.block, w.hq, w.hkv, w.head_dim, cap,
                                                   dt_code), dtype=torch.uint8, device=dev)
    a_ws = torch.zeros(max(1, sd.sd_spec_accept_workspace_size(w.batch, w.block, w.vocab, amode)),
                       dtype=torch.uint8, device=dev)
    lm_rows = lm["hidden"].shape[0]
    lm_out = torch.empty((lm_rows, w.vocab), dtype=torch.float32, device=dev)
    lm_ws = torch.zeros(sd.sd_lm_head_workspace_size(lm_rows, w.lm_width, w.vocab, dt_code),
                        dtype=torch.uint8, device=dev)
    n_out = torch.empty((w.batch,), dtype=torch.int32, device=dev)
    t_out = torch.empty((w.batch, w.block + 1), dtype=torch.int32, device=dev)
    al_ws = torch.zeros(sd.sd_spec_accept_logits_workspace_size(w.batch, w.block, w.vocab, amode),
                        dtype=torch.uint8, device=dev)
    nl_out = torch.empty((w.batch,), dtype=torch.int32, device=dev)
    dB, dr_rows, dd, _, _, dI, dL = synth.draft_dims(w)
    d_out = torch.empty((dB, dr_rows, dd), dtype=torch.float32, device=dev)
    d_ws = torch.zeros(sd.sd_semi_ar_layer_workspace_size(dB, dr_rows, dd, dr["hq"], dr["hkv"], dI, dL),
                       dtype=torch.uint8, device=dev)
    tl_out = torch.empty((w.batch, w.block + 1), dtype=torch.int32, device=dev)
    scale = 1.0 / math.sqrt(w.head_dim)

    # one drafting round in pipeline order: the draft side (compression of
    # the visual features, the draft layer step), then the target side
    # (verification attention, LM head, acceptance)
    def step(ev=None):
        if ev is not None:
            ev[0].record()
        sd.sd_latent_compress(lat_d, feats_d, w.c_heads, 1.0, out=c_out, workspace=c_ws)
        if ev is not None:
            ev[1].record()
        # the draft step writes the same cache slots every time (same positions)
        sd.sd_semi_ar_layer(du_d, dw_d, dkc_d, dvc_d, dpos_d, dr["hq"], dr["hkv"], dr["eps"],
                            dr["theta"], out=d_out, workspace=d_ws)
        if ev is not None:
            ev[6].record()
        sd.sd_verify_attention(q_d, k_d, v_d, kl_d, scale=scale, page_table=pt_d, out=v_out,
                               lse=v_lse, workspace=v_ws)
        if ev is not None:
            ev[2].record()
        sd.sd_lm_head_probs(h_d, wt_d, lm["temperature"], out=lm_out, workspace=lm_ws)
        if ev is not None:
            ev[3].record()
        sd.sd_spec_accept(p_d, qq_d, dr_d, u_d, amode, n_accepted=n_out, tokens=t_out,
                          workspace=a_ws)
        if ev is not None:
            ev[4].record()
        sd.sd_spec_accept_logits(zt_d, zd_d, drl_d, accl["philox_seed"], accl["philox_offset"],
                                 accl["temperature"], amode, n_accepted=nl_out, tokens=tl_out,
                                 workspace=al_ws)
        if ev is not None:
            ev[5].record()

    if args.copy_calibration_mib:
        src = torch.empty(args.copy_calibration_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # K drafts in K / k' passes (k' = K / 2): timed on its own, outside the
    # step (it repeats the draft layer and the LM head per pass); the head
    # weight doubles as the (tied) token embeddings
    kp = w.block // 2 if w.block % 2 == 0 else w.block
    rng = np.random.default_rng(w.seed)
    ph_np = rng.normal(size=2 * dd).astype(np.float32)
    u0_np = dr["u"].values[:, :1 + kp].copy()
    u0_np[:, 1:] = ph_np
    u0_d = to_dev(synth.Tensor(u0_np, "bf16"), dev)
    ph_d = to_dev(synth.Tensor(ph_np, "bf16"), dev)
    uk_d = torch.from_numpy((rng.integers(0, 1 << 24, size=(dB, w.block)) * 2.0 ** -24).astype(np.float32)).to(dev)
    kp_ws = torch.zeros(sd.sd_semi_ar_draft_workspace_size(dB, 1 + kp, dd, dr["hq"], dr["hkv"], dI, dL, w.vocab,
                                                           w.block, kp), dtype=torch.uint8, device=dev)
    kp_tok = torch.empty((dB, w.block), dtype=torch.int32, device=dev)
    kp_q = torch.empty((dB, w.block, w.vocab), dtype=torch.float32, device=dev)

    def kp_call():
        sd.sd_semi_ar_draft(u0_d, dw_d, wt_d, wt_d, ph_d, dkc_d, dvc_d, dpos_d, uk_d, w.block, kp, dr["hq"],
                            dr["hkv"], dr["eps"], dr["theta"], lm["temperature"], tokens=kp_tok, q=kp_q,
                            workspace=kp_ws)

    # the K / k' drafts and the int8 draft take bf16 weights only
    t_kp = t_q8 = None
    if w.dtype == "bf16":
        for _ in range(2):
            kp_call()
        kp_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(10)]
        for e in kp_ev:
            e[0].record()
            kp_call()
            e[1].record()
        torch.cuda.synchronize()
        t_kp = float(np.mean([e[0].elapsed_time(e[1]) for e in kp_ev]))
        kp_bytes = synth.draft_kp_bytes(w, kp)

    if w.dtype == "bf16":
        # the int8 draft's step (weight-only int8 rows), also timed on its own
        dq = synth.draft_inputs(w, q8=True)
        dq_w = {k: (to_dev(v, dev) if hasattr(v, "bits") else torch.from_numpy(v).to(dev))
                for k, v in dq["weights"].items()}
        dq_out = torch.empty_like(d_out)

        def q8_call():
            sd.sd_semi_ar_layer_q8(du_d, dq_w, dkc_d, dvc_d, dpos_d, dr["hq"], dr["hkv"], dr["eps"], dr["theta"],
                                   out=dq_out, workspace=d_ws)

        for _ in range(2):
            q8_call()
        q8_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(10)]
        for e in q8_ev:
            e[0].record()
            q8_call()
            e[1].record()
        torch.cuda.synchronize()
        t_q8 = float(np.mean([e[0].elapsed_time(e[1]) for e in q8_ev]))
        q8_bytes = synth.draft_q8_bytes(w)
        del dq_w

    # the average-pooling compressor on the compression's input, timed on its own
    ap_out = torch.empty_like(c_out)
    for _ in range(2):
        sd.sd_avg_pool_compress(feats_d, w.c_latents, out=ap_out)
    ap_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(10)]
    for e in ap_ev:
        e[0].record()
        sd.sd_avg_pool_compress(feats_d, w.c_latents, out=ap_out)
        e[1].record()
    torch.cuda.synchronize()
    t_ap = float(np.mean([e[0].elapsed_time(e[1]) for e in ap_ev]))
    es = 2 if w.dtype == "bf16" else 4
    ap_bytes = w.c_batch * w.c_tokens * w.c_width * es + w.c_batch * w.c_latents * w.c_width * 4

    # the int8 draft's compressor (int8 rows with power-of-two scales), timed
    # on its own on the same features quantised
    t_q8c = None
    if w.dtype == "bf16":
        qc = synth.compress_q8_inputs(w)
        qcd = {k_: torch.from_numpy(v_).to(dev) for k_, v_ in qc.items()}
        del qc
        n8 = sd.sd_latent_compress_q8_workspace_size(w.c_batch, w.c_tokens, w.c_latents, w.c_width, w.c_heads)
        ws8 = torch.zeros(max(n8, 1), dtype=torch.uint8, device=dev)
        q8c_out = torch.empty_like(c_out)

        def q8c_call():
            sd.sd_latent_compress_q8(qcd["latents_q"], qcd["latent_exp"], qcd["feats_q"], qcd["feat_exp"],
                                     w.c_heads, 1.0, out=q8c_out, workspace=ws8)

        for _ in range(2):
            q8c_call()
        q8c_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(10)]
        for e in q8c_ev:
            e[0].record()
            q8c_call()
            e[1].record()
        torch.cuda.synchronize()
        t_q8c = float(np.mean([e[0].elapsed_time(e[1]) for e in q8c_ev]))
        del qcd, ws8, q8c_out

    comp_ms = np.array([e[0].elapsed_time(e[1]) for e in events])
    ver_ms = np.array([e[6].elapsed_time(e[2]) for e in events])
    lm_ms = np.array([e[2].elapsed_time(e[3]) for e in events])
    acc_ms = np.array([e[3].elapsed_time(e[4]) for e in events])
    accl_ms = np.array([e[4].elapsed_time(e[5]) for e in events])
    draft_ms = np.array([e[1].elapsed_time(e[6]) for e in events])

    kv_bytes = synth.verify_kv_bytes(w, ver["kv_len"])
    flops = synth.compress_flops(w)
    c_bytes = synth.compress_bytes(w)
    n_host = n_out.cpu().numpy()
    a_bytes = accept_bytes(acc["p"], n_host)
    # Rooflines use each kernel's mean duration over the timed steps (the
    # figure a rocprofv3 kernel trace averages); `ops` adds medians and the
    # p10 / p90 spread, and `value` is taken at the medians.
    t_c, t_v, t_a = float(comp_ms.mean()), float(ver_ms.mean()), float(acc_ms.mean())
    t_l = float(lm_ms.mean())
    t_al = float(accl_ms.mean())
    t_d = float(draft_ms.mean())
    ops = {"latent_compress": op_stats(comp_ms), "verify_attention": op_stats(ver_ms),
           "spec_accept": op_stats(acc_ms), "lm_head": op_stats(lm_ms),
           "spec_accept_logits": op_stats(accl_ms), "semi_ar_layer": op_stats(draft_ms),
           "verify_step": op_stats(ver_ms + acc_ms)}
    d_bytes = synth.draft_bytes(w)
    al_bytes = accept_logits_bytes(w, nl_out.cpu().numpy())
    l_bytes = synth.lm_bytes(w, lm_rows)
    verify_step_ms = ops["verify_step"]["median_us"] * 1e-3
    value = kv_bytes / (verify_step_ms * 1e-3) / 1e12

    peak_c = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_VALU_PEAK_TFLOPS
    rl = {
        "latent_compress": {"bound": "mfma", "achieved": flops / (t_c * 1e-3) / 1e12,
                            "peak": peak_c, "unit": "TFLOP/s", "traffic": None,
                            "algorithmic": flops, "us": t_c * 1e3,
                            "hbm_gbs": c_bytes / (t_c * 1e-3) / 1e9},
        "verify_attention": {"bound": "hbm", "achieved": kv_bytes / (t_v * 1e-3) / 1e9,
                             "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None,
                             "algorithmic": kv_bytes, "us": t_v * 1e3},
        "spec_accept": {"bound": "hbm", "achieved": a_bytes / (t_a * 1e-3) / 1e9,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None,
                        "algorithmic": a_bytes, "us": t_a * 1e3},
        "lm_head": {"bound": "hbm", "achieved": l_bytes / (t_l * 1e-3) / 1e9,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None,
                    "algorithmic": l_bytes, "us": t_l * 1e3},
        "spec_accept_logits": {"bound": "hbm", "achieved": al_bytes / (t_al * 1e-3) / 1e9,
                               "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None,
                               "algorithmic": al_bytes, "us": t_al * 1e3},
        "semi_ar_layer": {"bound": "hbm", "achieved": d_bytes / (t_d * 1e-3) / 1e9,
                          "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None,
                          "algorithmic": d_bytes, "us": t_d * 1e3},
    }
    traffic = counter_traffic(w.name)
    for name_, r in rl.items():
        r["frac"] = r["achieved"] / r["peak"]
        r["traffic"] = traffic.get(name_)
    dominant = max(rl, key=lambda k_: rl[k_]["us"])     # the step's operations only
    if t_kp is not None:
        rl["semi_ar_draft_kp"] = {"bound": "hbm", "achieved": kp_bytes / (t_kp * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "traffic": None, "algorithmic": kp_bytes, "us": t_kp * 1e3,
                                  "frac": kp_bytes / (t_kp * 1e-3) / 1e9 / HBM_PEAK_GBS, "k_prime": kp,
                                  "drafts": w.block, "outside_step": True}
        rl["semi_ar_layer_q8"] = {"bound": "hbm", "achieved": q8_bytes / (t_q8 * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "traffic": None, "algorithmic": q8_bytes, "us": t_q8 * 1e3,
                                  "frac": q8_bytes / (t_q8 * 1e-3) / 1e9 / HBM_PEAK_GBS, "outside_step": True}
    if t_q8c is not None:
        fq8 = synth.compress_flops(w)
        rl["latent_compress_q8"] = {"bound": "mfma", "achieved": fq8 / (t_q8c * 1e-3) / 1e12,
                                    "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "traffic": None,
                                    "algorithmic": fq8, "us": t_q8c * 1e3,
                                    "frac": fq8 / (t_q8c * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                                    "hbm_gbs": synth.compress_q8_bytes(w) / (t_q8c * 1e-3) / 1e9,
                                    "outside_step": True}
    rl["avg_pool_compress"] = {"bound": "hbm", "achieved": ap_bytes / (t_ap * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                               "unit": "GB/s", "traffic": None, "algorithmic": ap_bytes, "us": t_ap * 1e3,
                               "frac": ap_bytes / (t_ap * 1e-3) / 1e9 / HBM_PEAK_GBS, "outside_step": True}
    roof = {k_: rl[dominant][k_] for k_ in ("bound", "achieved", "peak", "unit", "frac",
                                             "traffic")}
    roof["kernel"] = dominant

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "TB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": w.batch, "q_heads": w.hq, "kv_heads": w.hkv, "head_dim": w.head_dim,
            "kv_len": w.kv_len, "paged": w.paged, "block_k": w.block,
            "compress_tokens": w.c_tokens, "compress_width": w.c_width,
            "latents": w.c_latents, "compress_heads": w.c_heads,
            "vocab": w.vocab, "accept_mode": mode, "temperature": acc["temperature"],
            "lm_rows": lm_rows, "lm_width": w.lm_width,
            "draft_rows": dB * dr_rows, "draft_ffn": dI, "draft_ctx": w.draft_ctx,
        },
        "verify_step_us": verify_step_ms * 1e3,
        "verify_attention_us": ops["verify_attention"]["median_us"],
        "spec_accept_us": ops["spec_accept"]["median_us"],
        "latent_compress_us": ops["latent_compress"]["median_us"],
        "lm_head_us": t_l * 1e3,
        "lm_head_tbps": l_bytes / (t_l * 1e-3) / 1e12,
        "spec_accept_logits_us": t_al * 1e3,
        "semi_ar_layer_us": t_d * 1e3,
        "semi_ar_layer_tbps": d_bytes / (t_d * 1e-3) / 1e12,
        "semi_ar_draft_kp_us": t_kp * 1e3 if t_kp is not None else None,
        "semi_ar_layer_q8_us": t_q8 * 1e3 if t_q8 is not None else None,
        "avg_pool_compress_us": t_ap * 1e3,
        "latent_compress_q8_us": t_q8c * 1e3 if t_q8c is not None else None,
        "latent_compress_tflops": flops / (ops["latent_compress"]["median_us"] * 1e-6) / 1e12,
        "kv_read_tbps_attention_only": kv_bytes / (ops["verify_attention"]["median_us"] * 1e-6) / 1e12,
        "ops": ops,
        "timing": "value and the *_us figures: medians over the timed steps (HIP events on the "
                  "kernels' stream); ops: median, p10, p90, mean; rooflines: mean launch duration",
        "accepted_mean": float(n_host.mean()),
        "roofline": roof,
        "rooflines": rl,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        cb = cpu_baseline(w, comp, ver, acc, 0 if mode == "greedy" else 1, lm, accl, dr)
        cpu_step = cb["verify_s"] + cb["accept_s"]
        result["cpu_baseline"] = {
            "value": kv_bytes / cpu_step / 1e12, "unit": "TB/s", "cores": cb["threads"],
            "cpu_model": cb["cpu_model"], "kind": "oracle", "sample": cb["sample"],
            "verify_step_s": cpu_step, "latent_compress_s": cb["compress_s"],
            "lm_head_s": cb["lm_head_s"], "accept_logits_s": cb["accept_logits_s"],
            "draft_layer_s": cb["draft_layer_s"],
            "whole_step_s": cpu_step + cb["compress_s"] + cb["lm_head_s"] + cb["accept_logits_s"]
                            + cb["draft_layer_s"],
        }
    if not args.no_workloads:
        # the other workloads' compression, verification and acceptance in the
        # same run (the main workload's operations are in `ops`)
        wl = {}
        for other in synth.WORKLOADS:
            if other.name == w.name:
                continue
            print(f"[bench] timing workload {other.name}", file=sys.stderr, flush=True)
            wl[other.name] = time_workload_ops(other, dev, args.workload_steps, args.warmup)
        main_ = {"dtype": w.dtype, "accept_mode": mode}
        for name_, work_, unit_, peak_ in (("latent_compress", flops, "TFLOP/s", peak_c),
                                           ("verify_attention", kv_bytes, "GB/s", HBM_PEAK_GBS),
                                           ("spec_accept", a_bytes, "GB/s", HBM_PEAK_GBS)):
            st_ = dict(ops[name_])
            sc_ = 1e12 if unit_ == "TFLOP/s" else 1e9
            rate_ = work_ / (st_["median_us"] * 1e-6) / sc_
            st_.update({"algorithmic": work_, "unit": unit_, "achieved_at_median": rate_, "peak": peak_,
                        "frac_at_median": rate_ / peak_,
                        "frac_at_p90": work_ / (st_["p90_us"] * 1e-6) / sc_ / peak_})
            gate_ = GATES.get((w.name, name_))
            if gate_ is not None:
                st_["target_frac"] = gate_
                st_["target_met_at_median"] = bool(st_["frac_at_median"] >= gate_)
            main_[name_] = st_
        main_["verify_step"] = dict(ops["verify_step"])
        main_["verify_step"]["kv_read_tbps_at_median"] = value
        wl[w.name] = main_
        result["workloads"] = {o.name: wl[o.name] for o in synth.WORKLOADS if o.name in wl}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
