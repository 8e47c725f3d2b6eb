"""Throughput of the WitCert hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--tau T]

One step = one decode step of every layer of the workload, each layer running the
whole hot path on the GPU: the new token of every sequence written through the
dithered INT8 quantizer with its witness (and into the exact bf16 cache), the
metered decode attention over the INT8 cache, the gate at tau, and the exact
fallback for the routed KV heads.  The serving mix also writes one prefill
chunk per layer and step.  Caches are filled (prefill write, timed separately
as the quant+witness figure) and every decode-step input is generated on the
GPU before the timed region.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0       # MI355X HBM3E
# algorithmic bytes per token-head, set from the workload's shape in main(); at
# d = 128, B = 8: 128 + 128 codes, 2 + 2 scales, 16 witness = 276 (INT8), 272 (fp8),
# 512 (bf16), 260 (Tier B reads no witness), 512 in + 276 out for a bf16 write
INT8_BYTES = FP8_BYTES = BF16_BYTES = TIERB_BYTES = WRITE_BYTES_BF16_IN = 0
REPAIR_BUDGET = 64           # blocks per KV head that block repair may page in
DECODE_KERNEL_SRC = os.path.join(ROOT, "paper_2607_28699_amd", "csrc")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(DECODE_KERNEL_SRC)):
        with open(os.path.join(DECODE_KERNEL_SRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="gqa-28x4-d128-s32k-b4")
    ap.add_argument("--tau", type=float, default=0.2)
    ap.add_argument("--outlier-pairs", type=int, default=4,
                    help="bypassed RoPE pairs per KV head for the bypass measurement (0: skip it)")
    ap.add_argument("--tau-v", type=float, default=0.05, help="value-side threshold of the joint gate")
    ap.add_argument("--no-group-scales", dest="group_scales", action="store_false",
                    help="skip the measurement over caches with 32-channel group scales")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", dest="other_workloads", action="store_false",
                    help="skip the per-call figures of the 4k, 131k and serving workloads")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (HBM counter calibration)")
    return ap.parse_args()


def copy_calibration():
    import torch
    n = 1 << 28                     # 256 MiB each way
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_each_way": n, "launches": 3}), flush=True)


def make_timer(np, torch):
    """timed(fn, reps): fn(0) .. fn(reps - 1) captured back to back in one HIP graph,
    the graph replayed five times between events recorded on the launching stream;
    per-call milliseconds of each replay."""
    def timed(fn, reps, replays=5):
        fn(0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(reps):
                fn(i)
        g.replay()
        torch.cuda.synchronize()
        per_call = []
        for _ in range(replays):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            per_call.append(e0.elapsed_time(e1) / reps)
        del g
        return np.array(per_call)
    return timed


class Layout:
    """Slots of the decode sequences (and of the serving mix's prefill chunks)."""

    def __init__(self, wl, lens, extra_steps, np):
        self.lens = np.asarray(lens, dtype=np.int64)
        cap = self.lens + extra_steps
        chunk_cap = wl.chunk * extra_steps if wl.chunk else 0
        caps = np.concatenate([cap, [chunk_cap]]) if wl.chunk else cap
        import synth
        self.table, self.nblocks = synth.block_table(caps, permute=wl.ragged, seed_key=wl.wid)
        self.batch = len(lens)

    def slots(self, seq, positions, np):
        return self.table[seq, positions // 16].astype(np.int64) * 16 + positions % 16


def cpu_baseline(wl, lens, tau, seconds, np, torch):
    """The oracle, as it stands, on a bounded sample of the same workload: per
    sampled (sequence, layer), write the new token, metered decode over the
    sequence, gate, exact fallback.  Prefill quantization of the sample is not timed."""
    import threadpoolctl

    from oracle import decode as odec
    from oracle import gate as ogate
    from synth import torch_gen
    sm = 1.0 / np.sqrt(wl.d)
    timed, tokens, samples = 0.0, 0, 0
    layer_ids = list(range(wl.n_layers))
    for i in range(256):
        seq = i % len(lens)
        layer = layer_ids[(i * 7) % len(layer_ids)]
        L = int(lens[seq])
        pos = torch.arange(L, device="cuda")
        k, v = torch_gen.gen_kv_layer(wl, layer, seq, pos)
        kn, vn = torch_gen.gen_kv_layer(wl, layer, seq, torch.tensor([L], device="cuda"), step=0)
        q = torch_gen.gen_q_batch(wl, layer, 0, torch.tensor([L], device="cuda"))[0]
        k, v, kn, vn, q = (x.float().cpu().numpy().astype(np.float64) for x in (k, v, kn, vn, q))
        slots = np.arange(L + 1, dtype=np.int64)
        cache = odec.write_cache("int8_dither", k, v, slots[:L], layer, wl.philox_seed(), wl.bands,
                                 wl.rope_layout)
        t0 = time.perf_counter()
        new = odec.write_cache("int8_dither", kn, vn, slots[L:], layer, wl.philox_seed(), wl.bands,
                               wl.rope_layout)
        kh = np.concatenate([cache["khat"], new["khat"]])
        vh = np.concatenate([cache["vhat"], new["vhat"]])
        kw = np.concatenate([cache["kw"], new["kw"]])
        res = odec.metered_decode(q, kh, vh, kw, sm, wl.bands, wl.rope_layout)
        mq = ogate.gate_q(res["meter"], res["raw"], tau)
        mkv = ogate.gate_kv(mq[None], wl.group)[0]
        ex = odec.exact_decode(q, np.concatenate([k, kn]), np.concatenate([v, vn]), sm)
        _ = ogate.apply_fallback(res["out"], ex["out"], mkv, wl.group)
        timed += time.perf_counter() - t0
        tokens += L + 1
        samples += 1
        if timed >= seconds:
            break
    info = threadpoolctl.threadpool_info()
    blas = max([p.get("num_threads", 1) for p in info if p.get("user_api") == "blas"] or [1])
    # the same cell on one core (BLAS limited to one thread): the single-core figure
    one_t, one_tok = 0.0, 0
    with threadpoolctl.threadpool_limits(limits=1):
        while one_t < min(seconds / 4, 5.0):
            t0 = time.perf_counter()
            new = odec.write_cache("int8_dither", kn, vn, slots[L:], layer, wl.philox_seed(), wl.bands,
                                   wl.rope_layout)
            res = odec.metered_decode(q, np.concatenate([cache["khat"], new["khat"]]),
                                      np.concatenate([cache["vhat"], new["vhat"]]),
                                      np.concatenate([cache["kw"], new["kw"]]), sm, wl.bands, wl.rope_layout)
            mq = ogate.gate_q(res["meter"], res["raw"], tau)
            ex = odec.exact_decode(q, np.concatenate([k, kn]), np.concatenate([v, vn]), sm)
            _ = ogate.apply_fallback(res["out"], ex["out"], ogate.gate_kv(mq[None], wl.group)[0], wl.group)
            one_t += time.perf_counter() - t0
            one_tok += L + 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"value": tokens / timed, "unit": "KV tokens/s", "cores": int(blas), "kind": "oracle",
            "os_cpu_count": os.cpu_count(), "affinity_cpus": affinity, "blas_threads": int(blas),
            "single_core_value": one_tok / one_t,
            "sample": (f"{samples} (sequence, layer) cells at context {int(lens[0])}: new-token write, "
                       f"metered decode of all {wl.n_q} query heads, gate at tau={tau}, exact fallback; "
                       f"{timed:.1f} s of oracle time (float64 numpy; BLAS threads={blas}, "
                       f"elementwise single-threaded); single_core_value: the last cell again with "
                       f"BLAS limited to one thread for {one_t:.1f} s")}


# distinct layer caches per other workload: enough that the captured calls read
# well past the 256 MB MALL (4k x 8: 36 MB per layer; 131k x 1: 145 MB; serving: 550 MB)
OTHER_WORKLOADS = {"gqa-28x4-d128-s4k-b8": 28, "gqa-28x4-d128-s131k-b1": 8, "serving-64seq-paged": 2}


def other_workload(name, n_layers, tau, timed, np, torch):
    """Per-call figures of another workload's hot path: the metered INT8 decode with
    the gate, the exact fallback of the KV heads it routes, and the prefill write
    (quant + witness + exact copy); each call captured back to back over distinct
    layer caches and timed from graph replays, as for the main workload."""
    import paper_2607_28699_amd as wc
    import synth
    from synth import torch_gen
    wl = synth.WORKLOADS[name]
    dev = "cuda"
    lens = (synth.serving_lengths(wl.batch, wl.len_lo, wl.ctx) if wl.ragged
            else np.full(wl.batch, wl.ctx, dtype=np.int64))
    lay = Layout(wl.replace(chunk=0), lens, 0, np)
    caches, exact, qs = [], [], []
    wr_in = None
    for layer in range(n_layers):
        c = wc.PagedCache("int8_dither", lay.nblocks, wl.n_kv, wl.d, wl.bands, layer=layer,
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout)
        e = wc.PagedCache("bf16", lay.nblocks, wl.n_kv, wl.d, 0, layer=layer)
        ks, vs, ss = [], [], []
        for b in range(lay.batch):
            k, v = torch_gen.gen_kv_layer(wl, layer, b, torch.arange(int(lens[b]), device=dev))
            ks.append(k)
            vs.append(v)
            ss.append(torch.from_numpy(lay.slots(b, np.arange(int(lens[b])), np)).to(dev))
        k, v, sl = torch.cat(ks), torch.cat(vs), torch.cat(ss)
        wc.quantize_write_pair(c, e, k, v, sl)
        if layer == 0:
            wr_in = (k, v, sl)
        del ks, vs
        caches.append(c)
        exact.append(e)
        qs.append(torch_gen.gen_q_batch(wl, layer, 0, torch.from_numpy(lens - 1).to(dev)))
    torch.cuda.synchronize()
    table = torch.from_numpy(lay.table).to(dev)
    seq_lens = torch.from_numpy(lens.astype(np.int32)).to(dev)
    L = int(lens.max())
    ST = wc.split_tokens_for(lay.batch, wl.n_kv, L, total_tokens=int(lens.sum()))
    ws = wc.decode_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, L, ST)
    out = torch.empty((lay.batch, wl.n_q, wl.d), dtype=torch.bfloat16, device=dev)
    meter = torch.empty((lay.batch, wl.n_q), dtype=torch.float32, device=dev)
    raw = torch.empty_like(meter)
    mask_q = torch.empty((lay.batch, wl.n_q), dtype=torch.uint8, device=dev)
    mask_kv = torch.empty((lay.batch, wl.n_kv), dtype=torch.uint8, device=dev)
    sm = 1.0 / np.sqrt(wl.d)
    reps = 56
    dec_ms = float(np.median(timed(lambda i: wc.metered_decode_gate(
        caches[i % n_layers], qs[i % n_layers], table, seq_lens, L, sm, tau, ws=ws, split_tokens=ST, out=out,
        meter=meter, raw=raw, mask_q=mask_q, mask_kv=mask_kv), reps)))
    routed = float(mask_kv.float().mean().item())
    fb_ms = float(np.median(timed(lambda i: wc.exact_decode_attention(
        exact[i % n_layers], qs[i % n_layers], table, seq_lens, L, sm, mask_kv, out, ws=ws, split_tokens=ST),
        reps)))
    k, v, sl = wr_in
    wr_ms = float(np.median(timed(lambda i: wc.quantize_write_pair(caches[0], exact[0], k, v, sl), 4)))
    th = float(lens.sum()) * wl.n_kv                     # token-heads per call
    int8_b, bf16_b = 2 * wl.d + 4 + 2 * wl.bands, 4 * wl.d
    wr_b = 2 * wl.d * 2 + int8_b + bf16_b                 # bf16 K, V in; INT8 cache + exact copy out
    gb = lambda nbytes, ms: nbytes / (ms * 1e-3) / 1e9
    res = {"batch": lay.batch, "context": L, "mean_context": float(lens.mean()), "split_tokens": ST,
           "layer_caches": n_layers,
           "metered_decode": {"median_launch_ms": round(dec_ms, 4), "GBps": round(gb(th * int8_b, dec_ms), 1),
                              "frac_hbm": round(gb(th * int8_b, dec_ms) / HBM_PEAK_GBPS, 4),
                              "bytes_per_token_head": int8_b},
           "exact_fallback": {"median_launch_ms": round(fb_ms, 4), "routed_kv_fraction": routed,
                              "GBps": round(gb(th * routed * bf16_b, fb_ms), 1),
                              "frac_hbm": round(gb(th * routed * bf16_b, fb_ms) / HBM_PEAK_GBPS, 4)},
           "write_pair": {"median_launch_ms": round(wr_ms, 4), "token_heads": int(k.shape[0] * wl.n_kv),
                          "bytes_per_token_head": wr_b,
                          "GBps": round(gb(k.shape[0] * wl.n_kv * wr_b, wr_ms), 1),
                          "frac_hbm": round(gb(k.shape[0] * wl.n_kv * wr_b, wr_ms) / HBM_PEAK_GBPS, 4)}}
    del caches, exact, qs, ws, wr_in
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path would shard by sequence and KV head, one process per GPU, "
              "with no communication inside a layer's decode)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if args.copy_calibration:
        copy_calibration()
        return

    import paper_2607_28699_amd as wc
    import synth
    from synth import torch_gen

    wl = synth.WORKLOADS[args.workload]
    global INT8_BYTES, FP8_BYTES, BF16_BYTES, TIERB_BYTES, WRITE_BYTES_BF16_IN
    INT8_BYTES = 2 * wl.d + 4 + 2 * wl.bands
    FP8_BYTES = 2 * wl.d + 2 * wl.bands
    BF16_BYTES = 4 * wl.d
    TIERB_BYTES = INT8_BYTES - 2 * wl.bands
    WRITE_BYTES_BF16_IN = 2 * wl.d * (4 if wl.dtype == "f32" else 2) + INT8_BYTES   # inputs in, cache out
    dev = "cuda"
    K, W = args.steps, args.warmup
    lens0 = (synth.serving_lengths(wl.batch, wl.len_lo, wl.ctx) if wl.ragged
             else np.full(wl.batch, wl.ctx, dtype=np.int64))
    lay = Layout(wl, lens0, K + W, np)
    sm = 1.0 / np.sqrt(wl.d)
    seed = wl.philox_seed()

    # ---- caches and prefill write (timed separately: quant+witness throughput) ----
    # With --outlier-pairs m > 0 every layer also gets an INT8 cache whose keys
    # bypass the m RoPE pairs of largest energy over the layer's prefill keys (the
    # fixed per-(layer, KV head) set of the outlier-pair bypass), chosen on the GPU.
    caches, exact, byp_caches, gs_caches, fp8_caches = [], [], [], [], []
    gen0 = None
    m_byp = args.outlier_pairs
    for layer in range(wl.n_layers):
        c = wc.PagedCache("int8_dither", lay.nblocks, wl.n_kv, wl.d, wl.bands, layer=layer, seed=seed,
                          rope_layout=wl.rope_layout)
        e = wc.PagedCache("bf16", lay.nblocks, wl.n_kv, wl.d, 0, layer=layer)
        gen = []
        for b in range(lay.batch):
            L = int(lens0[b])
            k, v = torch_gen.gen_kv_layer(wl, layer, b, torch.arange(L, device=dev))
            gen.append((k, v, torch.from_numpy(lay.slots(b, np.arange(L), np)).to(dev)))
        f8 = wc.PagedCache("fp8_raw", lay.nblocks, wl.n_kv, wl.d, wl.bands, layer=layer,
                           rope_layout=wl.rope_layout)   # the second black-box quantizer
        for k, v, sl in gen:
            wc.quantize_write(c, k, v, sl)
            wc.quantize_write(e, k, v, sl)
            wc.quantize_write(f8, k, v, sl)
        fp8_caches.append(f8)
        if m_byp:
            cb = wc.PagedCache("int8_dither", lay.nblocks, wl.n_kv, wl.d, wl.bands, layer=layer, seed=seed,
                               rope_layout=wl.rope_layout, n_outlier_pairs=m_byp, value_side=True)
            cb.set_outlier_pairs(wc.select_outlier_pairs(torch.cat([k for k, _, _ in gen]), m_byp,
                                                         wl.rope_layout))
            for k, v, sl in gen:
                wc.quantize_write(cb, k, v, sl)
            byp_caches.append(cb)
            if args.group_scales:   # the same bypass with per-32-channel group scales
                cg = wc.PagedCache("int8_dither", lay.nblocks, wl.n_kv, wl.d, wl.bands, layer=layer,
                                   seed=seed, rope_layout=wl.rope_layout, n_outlier_pairs=m_byp,
                                   value_side=True, group_scales=True)
                cg.set_outlier_pairs(cb.tensors["outlier_pairs"])
                for k, v, sl in gen:
                    wc.quantize_write(cg, k, v, sl)
                gs_caches.append(cg)
        torch.cuda.synchronize()
        caches.append(c)
        exact.append(e)
        if layer == 0:
            gen0 = gen            # kept for timing the quantizing write below
        del gen
    torch.cuda.synchronize()

    # ---- decode-step inputs, resident before timing ----
    steps_in = []
    table = torch.from_numpy(lay.table).to(dev)
    for s in range(K + W):
        pos = torch.from_numpy(lens0 + s).to(dev)
        lens = torch.from_numpy((lens0 + s + 1).astype(np.int32)).to(dev)
        slots = torch.from_numpy(np.array([lay.slots(b, np.array([lens0[b] + s]), np)[0]
                                           for b in range(lay.batch)], dtype=np.int64)).to(dev)
        per_layer = []
        for layer in range(wl.n_layers):
            q = torch_gen.gen_q_batch(wl, layer, s, pos)
            kv = [torch_gen.gen_kv_layer(wl, layer, b, pos[b:b + 1], step=s) for b in range(lay.batch)]
            kn = torch.cat([x[0] for x in kv])
            vn = torch.cat([x[1] for x in kv])
            item = {"q": q, "k": kn, "v": vn}
            if wl.chunk:
                cpos = torch.arange(s * wl.chunk, (s + 1) * wl.chunk, device=dev)
                ck, cv = torch_gen.gen_kv_layer(wl, layer, lay.batch, cpos, step=s)
                item["ck"], item["cv"] = ck, cv
                item["cslots"] = torch.from_numpy(lay.slots(lay.batch, cpos.cpu().numpy(), np)).to(dev)
            per_layer.append(item)
        steps_in.append({"lens": lens, "slots": slots, "tokens": int((lens0 + s + 1).sum()),
                         "layers": per_layer})
    max_len_all = int(lens0.max() + K + W)
    # split length of every decode call, balanced over the batch's tokens (the host
    # knows the lengths; equal to the library default for equal lengths)
    ST = wc.split_tokens_for(lay.batch, wl.n_kv, max_len_all, total_tokens=int((lens0 + K + W).sum()))
    # the speculative step's split: its one launch holds the metered and the exact
    # workgroups, so about half as many splits fill the GPU once (its workspace needs
    # no more than the decode split's)
    ST_SPEC = wc.speculative_split_tokens(lay.batch, wl.n_kv, max_len_all, total_tokens=int((lens0 + K + W).sum()))
    ws = wc.decode_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, max_len_all, ST)
    ws_step = wc.certified_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, max_len_all, ST)
    out = torch.empty((lay.batch, wl.n_q, wl.d), dtype=torch.bfloat16, device=dev)
    meter = torch.empty((lay.batch, wl.n_q), dtype=torch.float32, device=dev)
    raw = torch.empty_like(meter)
    mask_q = torch.empty((lay.batch, wl.n_q), dtype=torch.uint8, device=dev)
    mask_kv = torch.empty((lay.batch, wl.n_kv), dtype=torch.uint8, device=dev)
    counts = torch.zeros(2, dtype=torch.int32, device=dev)

    def run_step(si, speculative):
        st = steps_in[si]
        step_call = wc.step_certified_decode_speculative if speculative else wc.step_certified_decode
        for layer in range(wl.n_layers):
            it = st["layers"][layer]
            # new tokens into the quantized cache and the exact bf16 copy in one pass
            if wl.chunk:
                wc.quantize_write_pair(caches[layer], exact[layer], it["ck"], it["cv"], it["cslots"])
            # the step's token of every sequence into the quantized cache and the exact
            # copy with the metered decode, the exact fallback (gated: its workgroups
            # decide their KV head's gate first; speculative: every KV head, beside the
            # metered decode) and one final merge
            step_call(caches[layer], exact[layer], it["k"], it["v"], st["slots"], it["q"],
                      table, st["lens"], max_len_all, sm, args.tau, ws=ws_step,
                      split_tokens=ST_SPEC if speculative else ST,
                      out=out, meter=meter, raw=raw, mask_q=mask_q, mask_kv=mask_kv, n_gated=counts)

    # The step form a serving loop would pick from what it observed: the speculative
    # one when the previous step's gate routed at least half of the KV heads (here:
    # the first step, run gated before the graphs are captured).
    counts.zero_()
    run_step(0, False)
    torch.cuda.synchronize()
    first_routed = float(counts[1].item()) / (wl.n_layers * lay.batch * wl.n_kv)
    speculative = first_routed >= 0.5
    # one decode step per HIP graph (all layers), replayed back to back: the timed
    # region is GPU work only, as in a graph-captured serving loop
    graphs = []
    for s in range(K + W):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run_step(s, speculative)
        graphs.append(g)
    for s in range(W):
        graphs[s].replay()
    torch.cuda.synchronize()
    counts.zero_()
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for s in range(K):
        graphs[W + s].replay()
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / K
    kv_tokens = sum(steps_in[W + s]["tokens"] for s in range(K)) * wl.n_layers
    value = kv_tokens / (total_ms / 1e3)
    gq, gkv = counts.cpu().tolist()
    frac_kv = gkv / (K * wl.n_layers * lay.batch * wl.n_kv)
    frac_q = gq / (K * wl.n_layers * lay.batch * wl.n_q)

    # ---- per-call timing: reps calls captured back to back in one HIP graph, the
    # replays timed with events on the launch stream (no host gaps between calls) ----
    timed = make_timer(np, torch)

    # quantize+witness write of the prefill: layer 0's sequences, each call
    # rewriting the same slots with the same values
    write_tokens = sum(k.shape[0] for k, _, _ in gen0) * wl.n_kv
    wr_ms = timed(lambda i: [wc.quantize_write(caches[0], k, v, sl) for k, v, sl in gen0], 4)
    write_ms = float(np.median(wr_ms))
    del gen0

    last = steps_in[W + K - 1]
    reps = 2 * wl.n_layers
    dec_ms = timed(lambda i: wc.metered_decode_gate(
        caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
        max_len_all, sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mask_q,
        mask_kv=mask_kv), reps)
    fb_ms = timed(lambda i: wc.exact_decode_attention(
        exact[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
        max_len_all, sm, mask_kv, out, ws=ws, split_tokens=ST), reps)
    routed = float(mask_kv.float().mean().item())    # the route mask the fallback timing used
    # the raw fp8 E4M3 cast (no scale) through the same meter: the decode-step tokens
    # as the timed steps wrote them, per-call time, and the gate fractions of both
    # quantizers at every tau of the sweep over the last step's layers (Tier A)
    for s_ in range(K + W):
        st_ = steps_in[s_]
        for layer in range(wl.n_layers):
            it = st_["layers"][layer]
            if wl.chunk:
                wc.quantize_write(fp8_caches[layer], it["ck"], it["cv"], it["cslots"])
            wc.quantize_write(fp8_caches[layer], it["k"], it["v"], st_["slots"])
    f8_ms = timed(lambda i: wc.metered_decode_gate(
        fp8_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
        max_len_all, sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mask_q,
        mask_kv=mask_kv), reps)
    taus = (0.05, 0.1, 0.2)
    sweep = {}
    for qname, cl in (("int8_dither", caches), ("fp8_raw", fp8_caches)):
        mets, raws_s = [], []
        for layer in range(wl.n_layers):
            wc.metered_decode_attention(cl[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                        sm, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw)
            mets.append(meter.clone())
            raws_s.append(raw.clone())
        mt_all, rw_all = torch.stack(mets), torch.stack(raws_s)     # [layers, batch, n_q]
        entry = {"raw_median": round(float(rw_all.median().item()), 4)}
        for tau in taus:
            gq_t = (mt_all > tau) if tau < 1 else (rw_all > tau)
            gkv_t = gq_t.view(wl.n_layers, lay.batch, wl.n_kv, wl.group).any(dim=-1)
            entry[f"tau_{tau}"] = {"fraction_q_heads": round(float(gq_t.float().mean().item()), 4),
                                   "fraction_kv_heads": round(float(gkv_t.float().mean().item()), 4)}
        sweep[qname] = entry
    # Tier-B certificate (Sec. 4.2) over the same caches: per-call time and, over
    # every layer of the last step, its gate fractions (delta_req 1e-2 over
    # layers x query heads x 256 steps)
    dloc = wc.tierb_delta_loc(1e-2, wl.n_layers, wl.n_q, 256)
    tb_ms = timed(lambda i: wc.tierb_decode_attention(
        caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
        max_len_all, sm, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw), reps)
    counts_b = torch.zeros(2, dtype=torch.int32, device=dev)
    mq_b, mkv_b = torch.empty_like(mask_q), torch.empty_like(mask_kv)
    for layer in range(wl.n_layers):
        wc.tierb_decode_attention(caches[layer], last["layers"][layer]["q"], table, last["lens"],
                                  max_len_all, sm, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw)
        wc.gate(meter, raw, wl.group, args.tau, n_gated=counts_b, mask_q=mq_b, mask_kv=mkv_b)
    gqb, gkvb = counts_b.cpu().tolist()

    # ---- outlier-pair bypass (Sec. 6.2): both certificates over caches whose keys
    # keep the m most energetic RoPE pairs in fp16, out of the amax ----
    byp = None
    if m_byp:
        for s in range(K + W):      # the decode-step tokens, as the timed steps wrote them
            st = steps_in[s]
            for layer in range(wl.n_layers):
                it = st["layers"][layer]
                for cc in ([byp_caches[layer]] + ([gs_caches[layer]] if gs_caches else [])):
                    if wl.chunk:
                        wc.quantize_write(cc, it["ck"], it["cv"], it["cslots"])
                    wc.quantize_write(cc, it["k"], it["v"], st["slots"])
        ba_ms = timed(lambda i: wc.metered_decode_gate(
            byp_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
            max_len_all, sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mask_q,
            mask_kv=mask_kv), reps)
        bb_ms = timed(lambda i: wc.tierb_decode_attention(
            byp_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
            max_len_all, sm, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw), reps)
        cnt = {"A": torch.zeros(2, dtype=torch.int32, device=dev), "B": torch.zeros(2, dtype=torch.int32, device=dev)}
        raws = {"A": [], "B": []}
        for layer in range(wl.n_layers):
            q_l = last["layers"][layer]["q"]
            wc.metered_decode_attention(byp_caches[layer], q_l, table, last["lens"], max_len_all, sm, ws=ws, split_tokens=ST,
                                        out=out, meter=meter, raw=raw)
            wc.gate(meter, raw, wl.group, args.tau, n_gated=cnt["A"], mask_q=mq_b, mask_kv=mkv_b)
            raws["A"].append(raw.clone())
            wc.tierb_decode_attention(byp_caches[layer], q_l, table, last["lens"], max_len_all, sm, dloc,
                                      ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw)
            wc.gate(meter, raw, wl.group, args.tau, n_gated=cnt["B"], mask_q=mq_b, mask_kv=mkv_b)
            raws["B"].append(raw.clone())
        # the fixed pair set itself: one layer's prefill keys, every KV head
        kcat = torch.cat([torch_gen.gen_kv_layer(wl, 0, b, torch.arange(int(lens0[b]), device=dev))[0]
                          for b in range(lay.batch)])
        pairs_out = torch.empty((wl.n_kv, m_byp), dtype=torch.int32, device=dev)
        sel_ws = torch.empty(wc.lib().wc_select_workspace_size(kcat.shape[0], wl.n_kv, wl.d),
                             dtype=torch.uint8, device=dev)
        sel_ms = float(np.median(timed(lambda i: wc.select_outlier_pairs(kcat, m_byp, wl.rope_layout,
                                                                         out=pairs_out, ws=sel_ws), 4)))
        n_cells = wl.n_layers * lay.batch
        byp = {"outlier_pairs": m_byp, "select_pairs": {
                   "median_launch_ms": round(sel_ms, 4), "rows": int(kcat.shape[0]),
                   "GBps": round(kcat.numel() * kcat.element_size() / (sel_ms * 1e-3) / 1e9, 1)}}
        for tier, ms, nbytes in (("tier_a", ba_ms, INT8_BYTES + 4 * m_byp), ("tier_b", bb_ms, TIERB_BYTES + 4 * m_byp)):
            key = "A" if tier == "tier_a" else "B"
            gq_, gkv_ = cnt[key].cpu().tolist()
            gbps = float(last["tokens"] * wl.n_kv) * nbytes / (float(np.median(ms)) * 1e-3) / 1e9
            byp[tier] = {"median_launch_ms": round(float(np.median(ms)), 4), "GBps": round(gbps, 1),
                         "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4), "bytes_per_token_head": nbytes,
                         "raw_median": round(float(torch.cat(raws[key]).median().item()), 4),
                         "gate_fraction_q_heads": round(gq_ / (n_cells * wl.n_q), 4),
                         "gate_fraction_kv_heads": round(gkv_ / (n_cells * wl.n_kv), 4)}
        del kcat

        # joint key + value certificate with its gate (Sec. 4.2 joint event) over the
        # same caches, Tier B keys at the same budget: the paper's deployment form
        mv = torch.empty_like(meter)
        jt_ms = timed(lambda i: wc.joint_decode_gate(
            byp_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
            max_len_all, sm, args.tau, args.tau_v, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, meter_v=mv,
            mask_q=mask_q, mask_kv=mask_kv), reps)
        cj = torch.zeros(2, dtype=torch.int32, device=dev)
        pass_k = pass_v = 0
        mvs = []
        for layer in range(wl.n_layers):
            wc.joint_decode_gate(byp_caches[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                 sm, args.tau, args.tau_v, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw,
                                 meter_v=mv, mask_q=mq_b, mask_kv=mkv_b, n_gated=cj)
            pass_k += int((meter <= args.tau).sum().item())
            pass_v += int((mv <= args.tau_v).sum().item())
            mvs.append(mv.clone())
        gqj, gkvj = cj.cpu().tolist()
        nbytes = TIERB_BYTES + 4 * m_byp + 4
        gbps = float(last["tokens"] * wl.n_kv) * nbytes / (float(np.median(jt_ms)) * 1e-3) / 1e9
        byp["joint"] = {"tier": "B", "tau_k": args.tau, "tau_v": args.tau_v,
                        "median_launch_ms": round(float(np.median(jt_ms)), 4), "GBps": round(gbps, 1),
                        "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4), "bytes_per_token_head": nbytes,
                        "meter_v_median": round(float(torch.cat(mvs).median().item()), 5),
                        "pass_k_fraction": round(pass_k / (n_cells * wl.n_q), 4),
                        "pass_v_fraction": round(pass_v / (n_cells * wl.n_q), 4),
                        "gate_fraction_q_heads": round(gqj / (n_cells * wl.n_q), 4),
                        "gate_fraction_kv_heads": round(gkvj / (n_cells * wl.n_kv), 4)}

        # block-granular repair (Sec. 6.3) of the KV heads the Tier-A gate routes over
        # the same caches: fixed 256-token blocks, paged in from
        # the exact bf16 cache in decreasing order of their meter shares until every
        # query head passes tau, at most REPAIR_BUDGET blocks per KV head.  Timed as
        # (metered decode + gate + repair) minus the metered decode + gate alone.
        nrep = torch.empty((lay.batch, wl.n_kv), dtype=torch.int32, device=dev)
        rlist = torch.empty((lay.batch, wl.n_kv, REPAIR_BUDGET), dtype=torch.int32, device=dev)
        rws = wc.repair_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, REPAIR_BUDGET)

        def dec_rep(i):
            layer = i % wl.n_layers
            q_l = last["layers"][layer]["q"]
            wc.metered_decode_gate(byp_caches[layer], q_l, table, last["lens"], max_len_all, sm, args.tau,
                                   ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b, mask_kv=mkv_b)
            wc.block_repair(byp_caches[layer], exact[layer], q_l, table, last["lens"], max_len_all, sm,
                            args.tau, ws, out, meter, raw, mkv_b, max_blocks=REPAIR_BUDGET, split_tokens=ST,
                            repaired=rlist, n_repaired=nrep, repair_ws=rws)
        dr_ms = timed(dec_rep, reps)
        nreps = []
        for layer in range(wl.n_layers):
            dec_rep(layer)
            nreps.append(nrep.clone())
        nr = torch.cat(nreps).flatten().cpu().numpy()
        routed_r = nr != 0
        fixed = nr > 0
        bs = 256   # repair blocks: fixed 256-token runs
        rep_ms = max(float(np.median(dr_ms)) - float(np.median(ba_ms)), 0.0)
        del rws
        whole = float(np.mean(last["lens"].cpu().numpy())) * BF16_BYTES
        byp["repair"] = {
            "tau": args.tau, "budget_blocks": REPAIR_BUDGET, "block_tokens": bs,
            "median_launch_ms": round(rep_ms, 4),
            "routed_kv_fraction": round(float(routed_r.mean()), 4),
            "repaired_fraction_of_routed": round(float(fixed.sum() / max(routed_r.sum(), 1)), 4),
            "median_blocks_repaired": float(np.median(nr[fixed])) if fixed.any() else None,
            "paged_bytes_per_repaired_kv_head": (round(float(np.median(nr[fixed])) * bs * BF16_BYTES)
                                                 if fixed.any() else None),
            "whole_head_bytes": round(whole)}

        # the exact store in host memory, as the paper's CPU copy (Sec. 6.3): two layers'
        # exact caches in pinned host memory, read by the kernels over the host link;
        # timed like the repair above: the whole-head fallback of the routed KV heads,
        # and block repair (each minus the metered decode + gate over the same caches)
        far_n = min(2, wl.n_layers)
        exact_h = [exact[layer].host_copy() for layer in range(far_n)]
        rws = wc.repair_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, REPAIR_BUDGET)

        def far_base(i):
            layer = i % far_n
            wc.metered_decode_gate(byp_caches[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                   sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b,
                                   mask_kv=mkv_b)

        def far_fallback(i):
            far_base(i)
            layer = i % far_n
            wc.exact_decode_attention(exact_h[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                      sm, mkv_b, out, ws=ws, split_tokens=ST)

        def far_repair(i):
            # block repair, then the whole-head fallback of the KV heads it left routed
            far_base(i)
            layer = i % far_n
            wc.block_repair(byp_caches[layer], exact_h[layer], last["layers"][layer]["q"], table, last["lens"],
                            max_len_all, sm, args.tau, ws, out, meter, raw, mkv_b, max_blocks=REPAIR_BUDGET,
                            split_tokens=ST, repaired=rlist, n_repaired=nrep, repair_ws=rws)
            wc.exact_decode_attention(exact_h[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                      sm, mkv_b, out, ws=ws, split_tokens=ST)
        fr = 2 * far_n
        fb0 = float(np.median(timed(far_base, fr)))
        ffb = max(float(np.median(timed(far_fallback, fr))) - fb0, 0.0)
        frp = max(float(np.median(timed(far_repair, fr))) - fb0, 0.0)
        nr_f = []
        for layer in range(far_n):
            far_repair(layer)
            nr_f.append(nrep.clone())
        nr_f = torch.cat(nr_f).flatten().cpu().numpy()
        fixed_f = nr_f > 0
        n_units = len(nr_f)
        byp["repair_host_store"] = {
            "layers": far_n, "exact_store": "pinned host memory, read by the kernels over the host link",
            "fallback_median_ms": round(ffb, 4), "repair_median_ms": round(frp, 4),
            "routed_kv_fraction": round(float((nr_f != 0).mean()), 4),
            "repaired_fraction_of_routed": round(float(fixed_f.sum() / max((nr_f != 0).sum(), 1)), 4),
            "exact_bytes_fallback": round(float((nr_f != 0).sum()) / n_units * lay.batch * wl.n_kv * whole),
            "exact_bytes_repair": round(float(nr_f[fixed_f].sum()) / n_units * lay.batch * wl.n_kv * bs * BF16_BYTES)}
        del exact_h, rws

        # group scales (Sec. 6.2 storage side, Table 4): the same bypass caches with one
        # fp16 scale per token and 32-channel group (8 bytes per side instead of 2),
        # both tiers with the fused gate, and their meters, on the matrix cores
        if gs_caches:
            ga_ms = timed(lambda i: wc.metered_decode_gate(
                gs_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
                max_len_all, sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b,
                mask_kv=mkv_b), reps)
            gb_ms = timed(lambda i: wc.tierb_decode_attention(
                gs_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
                max_len_all, sm, dloc, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw), reps)
            cnt_g = {"A": torch.zeros(2, dtype=torch.int32, device=dev),
                     "B": torch.zeros(2, dtype=torch.int32, device=dev)}
            raws_g = {"A": [], "B": []}
            for layer in range(wl.n_layers):
                q_l = last["layers"][layer]["q"]
                wc.metered_decode_attention(gs_caches[layer], q_l, table, last["lens"], max_len_all, sm,
                                            ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw)
                wc.gate(meter, raw, wl.group, args.tau, n_gated=cnt_g["A"], mask_q=mq_b, mask_kv=mkv_b)
                raws_g["A"].append(raw.clone())
                wc.tierb_decode_attention(gs_caches[layer], q_l, table, last["lens"], max_len_all, sm, dloc,
                                          ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw)
                wc.gate(meter, raw, wl.group, args.tau, n_gated=cnt_g["B"], mask_q=mq_b, mask_kv=mkv_b)
                raws_g["B"].append(raw.clone())
            gsd = {"path": "matrix cores (fp16 group scales)"}
            for tier, ms, nbytes in (("tier_a", ga_ms, INT8_BYTES + 4 * m_byp + 12),
                                     ("tier_b", gb_ms, TIERB_BYTES + 4 * m_byp + 12)):
                key = "A" if tier == "tier_a" else "B"
                gq_, gkv_ = cnt_g[key].cpu().tolist()
                gbps = float(last["tokens"] * wl.n_kv) * nbytes / (float(np.median(ms)) * 1e-3) / 1e9
                gsd[tier] = {"median_launch_ms": round(float(np.median(ms)), 4), "GBps": round(gbps, 1),
                             "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4), "bytes_per_token_head": nbytes,
                             "raw_median": round(float(torch.cat(raws_g[key]).median().item()), 4),
                             "gate_fraction_q_heads": round(gq_ / (n_cells * wl.n_q), 4),
                             "gate_fraction_kv_heads": round(gkv_ / (n_cells * wl.n_kv), 4)}
            byp["group_scales"] = gsd

        # incremental persistent repair (Sec. 6 gate; Sec. 6.3 gated evaluation (c)):
        # each layer's Tier-A decode, gate and block repair once more, then the write-back
        # (the taken blocks' pages, and every page of a KV head the budget left to the
        # whole-head fallback, are served from the exact store from then on); timed: the
        # next step's metered decode with the gate over the written-back caches, which
        # reads the marked pages as bf16 with bound 0
        for layer in range(wl.n_layers):
            byp_caches[layer].enable_repair(exact[layer])
        rws = wc.repair_workspace(lay.batch, wl.n_q, wl.n_kv, wl.d, REPAIR_BUDGET)
        for layer in range(wl.n_layers):
            q_l = last["layers"][layer]["q"]
            wc.metered_decode_gate(byp_caches[layer], q_l, table, last["lens"], max_len_all, sm, args.tau,
                                   ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b, mask_kv=mkv_b)
            wc.block_repair(byp_caches[layer], exact[layer], q_l, table, last["lens"], max_len_all, sm,
                            args.tau, ws, out, meter, raw, mkv_b, max_blocks=REPAIR_BUDGET, split_tokens=ST,
                            repaired=rlist, n_repaired=nrep, repair_ws=rws)
            wc.repair_write_back(byp_caches[layer], table, last["lens"], rlist, nrep, whole_kv=mkv_b)
        del rws
        pr_ms = timed(lambda i: wc.metered_decode_gate(
            byp_caches[i % wl.n_layers], last["layers"][i % wl.n_layers]["q"], table, last["lens"],
            max_len_all, sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b,
            mask_kv=mkv_b), reps)
        cnt_p = torch.zeros(2, dtype=torch.int32, device=dev)
        marked, pages_used = 0, 0
        used = torch.zeros(lay.nblocks, dtype=torch.bool, device=dev)
        for b in range(lay.batch):
            nb = (int(last["lens"][b].item()) + 15) // 16
            used[table[b, :nb].long()] = True
        for layer in range(wl.n_layers):
            wc.metered_decode_gate(byp_caches[layer], last["layers"][layer]["q"], table, last["lens"], max_len_all,
                                   sm, args.tau, ws=ws, split_tokens=ST, out=out, meter=meter, raw=raw, mask_q=mq_b,
                                   mask_kv=mkv_b, n_gated=cnt_p)
            mk_ = byp_caches[layer].tensors["repaired"][used]
            marked += int(mk_.sum().item())
            pages_used += int(mk_.numel())
        gqp, gkvp = cnt_p.cpu().tolist()
        byp["persistent_repair"] = {
            "tau": args.tau, "budget_blocks": REPAIR_BUDGET,
            "marked_page_fraction": round(marked / max(pages_used, 1), 4),
            "next_step_median_launch_ms": round(float(np.median(pr_ms)), 4),
            "next_step_gate_fraction_q_heads": round(gqp / (n_cells * wl.n_q), 4),
            "next_step_gate_fraction_kv_heads": round(gkvp / (n_cells * wl.n_kv), 4)}
    th_per_launch = float(last["tokens"] * wl.n_kv)
    tb_gbps = th_per_launch * TIERB_BYTES / (float(np.median(tb_ms)) * 1e-3) / 1e9
    dec_gbps = th_per_launch * INT8_BYTES / (float(np.median(dec_ms)) * 1e-3) / 1e9
    fb_bytes = th_per_launch * routed * BF16_BYTES
    fb_gbps = fb_bytes / (float(np.median(fb_ms)) * 1e-3) / 1e9 if routed > 0 else 0.0
    write_gbps = write_tokens * WRITE_BYTES_BF16_IN / (write_ms * 1e-3) / 1e9   # per prefill of one layer

    # The roofline object is the metric's kernel: the metered INT8 decode with its
    # fused gate (decode_mfma_kernel + merge_kernel), 276 algorithmic bytes per
    # token-head over the call's token-heads, per-call time from the event-timed
    # graph replays above.  The exact fallback gets an object of its own.
    def traffic_of(key):
        prof = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
        if not os.path.exists(prof):
            return None
        with open(prof) as fh:
            pj = json.load(fh)
        if pj.get("kernel_source_hash") != kernel_source_hash():
            return None
        return pj.get("bytes_per_launch", {}).get(key)

    roof = {"kernel": "metered INT8 decode with the gate (decode_mfma_kernel + merge_kernel)", "bound": "hbm",
            "achieved": round(dec_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(dec_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic_of("metered_decode"),
            "algorithmic_bytes_per_launch": th_per_launch * INT8_BYTES,
            "bytes_per_token_head": INT8_BYTES, "token_heads_per_launch": th_per_launch,
            "median_launch_ms": round(float(np.median(dec_ms)), 4)}
    roof_fb = {"kernel": "exact bf16 fallback (decode_mfma_kernel + merge_kernel)", "bound": "hbm",
               "achieved": round(fb_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
               "frac": round(fb_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic_of("exact_fallback"),
               "algorithmic_bytes_per_launch": fb_bytes, "bytes_per_token_head": BF16_BYTES,
               "routed_kv_fraction": routed, "median_launch_ms": round(float(np.median(fb_ms)), 4)}

    line = {
        "metric": "metered INT8 decode-attn KV tokens/s & HBM GB/s (% peak); quant+witness GB/s",
        "value": round(value, 1), "unit": "KV tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp16 MFMA operands (exact int8 codes and dither), fp32 accumulate; bf16 q, K/V inputs and out",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": wl.n_layers, "n_q": wl.n_q, "n_kv": wl.n_kv,
                   "head_dim": wl.d, "bands": wl.bands, "batch": lay.batch,
                   "context": int(lens0.max()), "mean_context": float(lens0.mean()),
                   "tau": args.tau, "split_tokens": ST, "step_split_tokens": ST_SPEC if speculative else ST,
                   "cache": "int8 dither + fp16 scales + fp16 key witness",
                   "fallback": "bf16 exact cache in HBM",
                   "step": ("certified, speculative (exact fallback of every KV head beside the metered decode, "
                            "gate in the final merge)" if speculative else
                            "certified, gated (exact fallback of the routed KV heads after the metered decode)"),
                   "first_step_routed_kv_fraction": round(first_routed, 4)},
        "roofline": roof,
        "roofline_exact_fallback": roof_fb,
        "value_note": ("KV tokens attended per second over whole decode steps; each step includes the bf16 "
                       "exact-fallback re-read of the routed KV heads (routed fraction in gate)"),
        "metered_decode": {"median_launch_ms": round(float(np.median(dec_ms)), 4), "GBps": round(dec_gbps, 1),
                           "frac_hbm": round(dec_gbps / HBM_PEAK_GBPS, 4),
                           "bytes_per_token_head": INT8_BYTES},
        "exact_fallback": {"median_launch_ms": round(float(np.median(fb_ms)), 4), "GBps": round(fb_gbps, 1),
                           "frac_hbm": round(fb_gbps / HBM_PEAK_GBPS, 4), "routed_kv_fraction": routed},
        "gate": {"tau": args.tau, "fraction_q_heads": round(frac_q, 4),
                 "fraction_kv_heads": round(frac_kv, 4)},
        "fp8_raw_decode": {"median_launch_ms": round(float(np.median(f8_ms)), 4),
                           "GBps": round(th_per_launch * FP8_BYTES / (float(np.median(f8_ms)) * 1e-3) / 1e9, 1),
                           "frac_hbm": round(th_per_launch * FP8_BYTES / (float(np.median(f8_ms)) * 1e-3) / 1e9
                                             / HBM_PEAK_GBPS, 4),
                           "bytes_per_token_head": FP8_BYTES},
        "gate_sweep": sweep,
        "kv_bytes_per_token": {"int8_dither": wl.n_layers * wl.n_kv * INT8_BYTES,
                               "fp8_raw": wl.n_layers * wl.n_kv * FP8_BYTES,
                               "bf16": wl.n_layers * wl.n_kv * BF16_BYTES},
        "tierb": {"median_launch_ms": round(float(np.median(tb_ms)), 4), "GBps": round(tb_gbps, 1),
                  "frac_hbm": round(tb_gbps / HBM_PEAK_GBPS, 4), "bytes_per_token_head": TIERB_BYTES,
                  "delta_req": 1e-2, "delta_loc": dloc,
                  "gate_fraction_q_heads": round(gqb / (wl.n_layers * lay.batch * wl.n_q), 4),
                  "gate_fraction_kv_heads": round(gkvb / (wl.n_layers * lay.batch * wl.n_kv), 4)},
        "bypass": byp,
        "quant_witness": {"GBps": round(write_gbps, 1), "frac_hbm": round(write_gbps / HBM_PEAK_GBPS, 4),
                          "bytes_per_token_head": WRITE_BYTES_BF16_IN,
                          "token_heads": write_tokens},
        "kernel_source_hash": kernel_source_hash(),
    }
    if args.other_workloads and args.workload == "gqa-28x4-d128-s32k-b4":
        # free the main workload's caches first
        del caches, exact, byp_caches, gs_caches, fp8_caches, graphs, steps_in
        torch.cuda.empty_cache()
        line["other_workloads"] = {n: other_workload(n, nl, args.tau, timed, np, torch)
                                   for n, nl in OTHER_WORKLOADS.items()}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, lens0, args.tau, args.cpu_seconds, np, torch)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
