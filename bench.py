#!/usr/bin/env python
"""GSRQ hot-path benchmark on one MI355X.

One step = for the K cache and then the V cache of one LLaMA-3-8B-shaped
layer (32768 tokens x 8 KV heads x 128, float16; synthetic, see synth.py):
weighted GSKM codebook learning (d=8, K=256, one stage, T=20 iterations with
the stop rule of Algorithm 1), then 1-bit GSRQ encode, then gather-sum decode
to float16.  Inputs are resident in HBM before timing starts.

Prints one JSON line.  `value` is vectors/s over the whole step (a vector is
one token's 128-element K or V row of one head); the per-kernel figures come
from HIP events recorded around each launch on its own stream during the
timed steps.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "GSRQ encode vectors/s + GSKM iter/s at 1-bit; % of MFMA / HBM roofline"
# HBM bytes per launch of each workload's dominant kernel, from the FETCH_SIZE /
# WRITE_SIZE rocprofv3 passes (profiles/hbm_traffic_<workload>.md, read counts
# scaled x2.000 and writes x1.000 against a 256 MiB reference copy).  Valid
# only for the kernel source those passes measured; other workloads: null.
TRAFFIC = {
    "llama3_8b_layer_1bit": {"source": "gsrq.hip", "source_sha256_prefix": "e3353425db29e5d4",
                             "bytes_per_launch": 116563529},
    "llama3_8b_cache_1bit": {"source": "gsrq.hip", "source_sha256_prefix": "e3353425db29e5d4",
                             "bytes_per_launch": 321209405},
    "large_codebook_d128": {"source": "gsrq_wide.hip", "source_sha256_prefix": "363b3302a7802544",
                            "bytes_per_launch": 334662782},
    "paper_rates_d128": {"source": "gsrq_wide.hip", "source_sha256_prefix": "bffb1448b9cbf9bf",
                         "bytes_per_launch": 141466069},
    "rate_sweep_d16": {"source": "gsrq_wide.hip", "source_sha256_prefix": "363b3302a7802544",
                       "bytes_per_launch": 289978206},
    "decode_attention_1bit": {"source": "gsrq_attn.hip", "source_sha256_prefix": "123617164b1ac182",
                              "bytes_per_launch": 89763895},
    "decode_attention_075bit": {"source": "gsrq_attn.hip",
                                "source_sha256_prefix": "123617164b1ac182",
                                "bytes_per_launch": 177580762},
}
PEAK_MFMA_F16_TFLOPS = 2500.0   # MI355X dense fp16 MFMA
PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E
PEAK_LDS_TBPS = 256 * 128 * 2.4e9 / 1e12   # LDS: 256 CUs x 128 B/clk x 2.4 GHz
HEAD_DIM = 128


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llama3_8b_layer_1bit")
    ap.add_argument("--stages", type=int, default=0,
                    help="override the workload's number of residual stages M")
    ap.add_argument("--cpu-groups", type=int, default=128,
                    help="subspaces of the K cache the CPU-baseline sample runs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the measurements outside the step (per-token weights, "
                         "appended-token encode), e.g. for kernel profiles of the step alone")
    ap.add_argument("--copy-ref-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(reference dispatch for scaling HBM counters)")
    return ap.parse_args()


def cpu_baseline(kv, wl, n_groups):
    """Time the float64 oracle on a bounded sample of the same step and scale
    it to vectors/s of the whole step."""
    import numpy as np
    from oracle import gsrq_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    X = kv.keys.astype(np.float64)
    w = kv.w_keys.astype(np.float64)
    d, K, T = wl.d, wl.K, wl.T
    t_init = t_iter = t_enc = t_dec = 0.0
    n_iter = 2
    for g in range(n_groups):
        Xg = X[:, g * d:(g + 1) * d]
        t0 = time.perf_counter()
        gain, shape, prev = O.gskm_init(Xg, w, kv.seeds_keys[0, g])
        t1 = time.perf_counter()
        for _ in range(n_iter):
            a = O.gskm_assign(Xg, gain, shape)
            gain, shape = O.gskm_update(Xg, w, a, gain, shape)
        t2 = time.perf_counter()
        codes, _ = O.gsrq_encode(Xg, gain[None, None], shape[None, None])
        t3 = time.perf_counter()
        O.gsrq_decode(codes, gain[None, None], shape[None, None])
        t4 = time.perf_counter()
        t_init += t1 - t0
        t_iter += (t2 - t1) / n_iter
        t_enc += t3 - t2
        t_dec += t4 - t3
    per_group = (t_init + T * t_iter + t_enc + t_dec) / n_groups
    step_s = 2 * wl.G * wl.M * per_group                # K and V, every subspace and stage
    vectors = 2 * wl.N * (wl.D // HEAD_DIM)
    sample_s = t_init + n_iter * t_iter + t_enc + t_dec
    return {
        "value": vectors / step_s, "unit": "vectors/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"float64 oracle on {n_groups} of {wl.G} K-cache subspaces of this workload: "
                   f"init + {n_iter} GSKM iterations + encode + decode each ({sample_s:.1f} s), "
                   f"scaled to {T} iterations, {wl.G} subspaces, {wl.M} stage(s) and both "
                   f"caches (K, V)"),
        "est_step_s": step_s,
    }


def measured_traffic(name):
    """HBM bytes per launch of the workload's dominant kernel from its
    committed counter summary, or None when its source has changed since."""
    import hashlib
    tr = TRAFFIC.get(name)
    if tr is None:
        return None
    src = os.path.join(ROOT, "paper_2607_01065_amd", "csrc", tr["source"])
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    return tr["bytes_per_launch"] if sha == tr["source_sha256_prefix"] else None


def cache_cpu_baseline(X, gain, shape, wl, budget_s=10.0, rows=32768):
    """The float64 oracle's encode + decode of one layer's key rows with the
    layer's codebook, on a bounded sample (the first `rows` tokens of as many
    subspaces as fit the time budget), scaled to vectors/s of the whole step
    (every layer, K and V, all tokens and subspaces)."""
    import numpy as np
    from oracle import gsrq_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    d, G = wl.d, wl.D // wl.d
    rows = min(rows, wl.N)
    Xs = X[:rows].float().cpu().numpy().astype(np.float64)
    gs = gain[0].cpu().numpy().astype(np.float64)
    ss = shape[0].cpu().numpy().astype(np.float64)
    spent, n = 0.0, 0
    while n < G and spent < budget_s:
        Xg = Xs[:, n * d:(n + 1) * d]
        t0 = time.perf_counter()
        codes, _ = O.gsrq_encode(Xg, gs[n][None, None], ss[n][None, None])
        O.gsrq_decode(codes, gs[n][None, None], ss[n][None, None])
        spent += time.perf_counter() - t0
        n += 1
    step_s = spent / (n * rows) * wl.N * G * 2 * wl.layers
    vectors = wl.layers * 2 * wl.N * (wl.D // HEAD_DIM)
    return {
        "value": vectors / step_s, "unit": "vectors/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"float64 oracle encode + decode of {rows} tokens of {n} of {G} key subspaces "
                   f"of layer 0 with the layer's codebook ({spent:.1f} s), scaled to "
                   f"{wl.N} tokens, {G} subspaces, K and V and {wl.layers} layers"),
        "est_step_s": step_s,
    }


def full_cache(args, wl):
    """Full-model cache: every layer's K and V codebooks are trained (T
    iterations, weighted) on a separate 4096-token calibration draw of the
    layer; the timed step encodes and decodes all layers' tokens, which are
    resident in HBM (drawn on the device) before timing starts."""
    import numpy as np
    import torch

    import synth
    from paper_2607_01065_amd import gsrq as B

    B.load_library()
    N, D, d, K, T, L = wl.N, wl.D, wl.d, wl.K, wl.T, wl.layers
    G = D // d
    heads = D // HEAD_DIM
    dev = torch.device("cuda", 0)
    ws_train = torch.empty(B.train_workspace_bytes(4096, D, d, K), dtype=torch.uint8, device=dev)
    ws_enc = torch.empty(B.encode_workspace_bytes(N, D, d, K, 1), dtype=torch.uint8, device=dev)
    W = B.code_words(N, D, d, K, 1)
    layers = []
    t0 = time.perf_counter()
    for layer in range(L):
        cal = synth.make_calibration(wl, layer, seed=0, N=4096, M=1)
        keys, values, _, _ = synth.make_kv_device(wl, layer, seed=0, device=dev)
        entry = []
        for X, Xc, wc, seeds in ((keys, cal.keys, cal.w_keys, cal.seeds_keys),
                                 (values, cal.values, cal.w_values, cal.seeds_values)):
            r = B.train_stage(torch.from_numpy(Xc).to(dev), d, K, T, seed_rows=seeds[0],
                              w=torch.from_numpy(wc).to(dev), trace=False, workspace=ws_train)
            entry.append(dict(X=X, gain=r.gain[None].contiguous(), shape=r.shape[None].contiguous(),
                              codes=torch.empty((N, W), dtype=torch.int32, device=dev)))
        layers.append(entry)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    xhat = torch.empty((N, D), dtype=torch.float16, device=dev)

    def step():
        for entry in layers:
            for c in entry:
                B.encode(c["X"], c["gain"], c["shape"], codes=c["codes"], workspace=ws_enc)
                B.decode(c["codes"], c["gain"], c["shape"], D, out=xhat)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # events only around the encoder launches inside the timed region; the
    # per-kernel breakdown comes from one instrumented step afterwards
    B.timing_enable(True, kinds=["encode"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step()
        if k == 0:
            B.timing_enable(False)   # records of the enqueued launches are kept
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    tim_timed = B.timing_read()
    tim = breakdown(B, step)
    tim["encode"] = tim_timed["encode"]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    vectors = L * 2 * N * heads

    def avg_us(kind):
        ms, n = tim[kind]
        return (ms / n * 1e3) if n else None

    e_us, dcd_us = avg_us("encode"), avg_us("decode")
    dec_bytes = N * G * np.log2(K) / 8 + N * D * 2
    out = {
        "metric": METRIC, "value": vectors / (ms_per_step / 1e3), "unit": "vectors/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "shape": wl.note, "layers": L, "tokens": N,
                   "kv_heads": heads, "head_dim": HEAD_DIM, "d": d, "K": K, "M": 1,
                   "calibration": "4096-token draw per layer, weighted GSKM T=%d" % T,
                   "caches": "K and V", "step": "encode + decode of every layer",
                   "bits_per_element": B.bits_per_element(d, K, 1)},
        "setup_s": setup_s,
        "encode_vectors_per_s": N * heads / (e_us * 1e-6),
        "decode_GBps": dec_bytes / (dcd_us * 1e-6) / 1e9,
        "decode_hbm_frac": dec_bytes / (dcd_us * 1e-6) / 1e9 / PEAK_HBM_GBPS,
        "kernels_us": {k: {"avg_us": avg_us(k), "launches": tim[k][1]} for k in tim},
        "kernels_us_source": "encode: HIP events around its launches in the first timed "
                             "step; others: one instrumented step after the timed region",
    }
    # the dominant kernel is the encoder (one launch per layer and cache):
    # eq. (5) scores of every row against every codeword, 2 N D K flops
    enc_flops = 2.0 * N * D * K
    achieved = enc_flops / (e_us * 1e-6) / 1e12
    out["roofline"] = {"kernel": "encode (eq. 5 scores + argmin + bit-pack, one stage)",
                       "bound": "mfma", "achieved": achieved, "peak": PEAK_MFMA_F16_TFLOPS,
                       "unit": "TFLOP/s", "frac": achieved / PEAK_MFMA_F16_TFLOPS,
                       "traffic": measured_traffic(wl.name),
                       "traffic_unit": "HBM bytes per launch", "flops_per_launch": enc_flops,
                       "avg_launch_us": e_us}
    if args.copy_ref_mib > 0:
        out["copy_ref_bytes"] = copy_reference(args.copy_ref_mib, dev)
    if not args.no_cpu_baseline:
        c = layers[0][0]
        out["cpu_baseline"] = cache_cpu_baseline(c["X"], c["gain"], c["shape"], wl)
    print(json.dumps(out), flush=True)


def extra_paths(B, cache, wl, dev, reps=50):
    """Measured after the timed region, outside `value`: per-token weights
    from gradient rows of the layer's shape (Sec. 5.3, Appendix B), the
    encode latency of a few appended tokens with the layer's trained codebook
    (the per-step append of autoregressive decoding), and one decoding step
    of attention over coded caches (Appendix C)."""
    import torch

    import synth
    out = {}
    G = torch.from_numpy(synth.gradient_rows(wl.N, wl.D, seed=1)).to(dev)
    B.row_weights(G)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        B.row_weights(G)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    out["row_weights"] = {"us": us, "tokens": wl.N, "grad_GBps": G.numel() * 2 / (us * 1e-6) / 1e9}
    del G
    app, app_p, app_k = {}, {}, {}
    prep = B.prepare_codebook(cache["gain"], cache["shape"]) if wl.d <= 8 and wl.K <= 256 else None
    for n in (1, 8, 64):
        X = cache["X"][:n].contiguous()
        codes = torch.empty((n, cache["codes"].shape[1]), dtype=torch.int32, device=dev)
        ws = torch.empty(B.encode_workspace_bytes(n, wl.D, wl.d, wl.K, wl.M), dtype=torch.uint8,
                         device=dev)
        B.encode(X, cache["gain"], cache["shape"], codes=codes, workspace=ws)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            B.encode(X, cache["gain"], cache["shape"], codes=codes, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        app[str(n)] = e0.elapsed_time(e1) / reps * 1e3
        if prep is not None:
            B.encode_prepared(X, prep, codes=codes)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                B.encode_prepared(X, prep, codes=codes)
            e1.record()
            torch.cuda.synchronize()
            app_p[str(n)] = e0.elapsed_time(e1) / reps * 1e3
            # kernel time alone (launch timing of the encode kind)
            B.timing_enable(True, kinds=["encode"])
            for _ in range(reps):
                B.encode_prepared(X, prep, codes=codes)
            B.timing_enable(False)
            ms, cnt = B.timing_read()["encode"]
            app_k[str(n)] = ms / max(cnt, 1) * 1e3
    out["append_encode_us"] = app
    if prep is not None:
        out["append_encode_prepared_us"] = app_p
        out["append_encode_prepared_kernel_us"] = app_k
    out.update(attention_measure(B, dev))
    return out


ATTN_SHAPE = dict(B=8, cap=32768, Hkv=8, GQ=4)   # LLaMA-3-8B heads, 32K-token context


ATTN_RQ_STAGES = 12   # the paper's 0.75-bit setting: d = 128, K = 256, 12 stages


def attention_measure(B, dev, reps=50, shape=ATTN_SHAPE, layout="1bit"):
    """One decoding step of attention over coded K/V caches
    (gsrq_attn_decode: unpack, dequantise, RoPE, attention) for 8 sequences
    of 32768 tokens, 32 query / 8 key-value heads, next to float16 attention
    over an already dequantised and rotated cache of the same shape (two
    float16 matmuls and a float32 softmax, reading 1.07 GB).  layout "1bit":
    d = 8, K = 256, one stage; "075bit": the paper's 0.75-bit residual
    coding, d = 128, K = 256, 12 stages (Sec. 6.2; Appendix C)."""
    import math

    import torch

    import synth
    Bn, cap, Hkv, GQ = shape["B"], shape["cap"], shape["Hkv"], shape["GQ"]
    Hq = Hkv * GQ
    rq = layout == "075bit"
    M = ATTN_RQ_STAGES if rq else 1
    if rq:
        case = synth.attn_case_rq(Bn, cap, [cap] * Bn, Hkv, GQ, M=M, seed=0, q_dtype="float16")
    else:
        case = synth.attn_case(Bn, cap, [cap] * Bn, Hkv, GQ, seed=0, q_dtype="float16")
    t = {k: torch.from_numpy(case[k]).to(dev) for k in
         ("k_codes", "v_codes", "lens", "k_gain", "k_shape", "v_gain", "v_shape", "q")}
    ws = torch.empty(B.attn_workspace_bytes(Bn, cap, Hq, Hkv, d=HEAD_DIM if rq else 8, M=M),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((Bn, Hq, HEAD_DIM), dtype=torch.float32, device=dev)

    def call():
        B.attn_decode(t["k_codes"], t["v_codes"], t["lens"], t["k_gain"], t["k_shape"],
                      t["v_gain"], t["v_shape"], t["q"], out=out, workspace=ws)

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    call_us = timed(call)

    def call_ready():
        B.attn_decode(t["k_codes"], t["v_codes"], t["lens"], t["k_gain"], t["k_shape"],
                      t["v_gain"], t["v_shape"], t["q"], out=out, workspace=ws,
                      tables_ready=True)

    ready_us = timed(call_ready)
    B.timing_enable(True, kinds=["attention"])
    timed(call)
    tim = B.timing_read()
    B.timing_enable(False)
    kern_us = tim["attention"][0] / tim["attention"][1] * 1e3
    tok_heads = Bn * cap * Hkv
    if rq:
        code_bytes = 2 * tok_heads * M               # one byte per stage, K and V
        cb_bytes = 2 * Hkv * M * 256 * 129 * 4       # both codebooks (gain + 128-element shape)
    else:
        code_bytes = 2 * tok_heads * 16              # 8-bit codes of 16 subspaces, K and V
        cb_bytes = 2 * Hkv * 16 * 256 * 9 * 4        # both codebooks (gain + 8-element shape)
    io_bytes = Bn * Hq * HEAD_DIM * (2 + 4)          # float16 queries in, float32 out
    alg_bytes = code_bytes + cb_bytes + io_bytes
    del t, ws, out, case
    # float16 attention over a dequantised, rotated cache of the same shape
    scale = 1.0 / math.sqrt(HEAD_DIM)
    kT = torch.randn((Bn * Hkv, HEAD_DIM, cap), dtype=torch.float16, device=dev)
    vf = torch.randn((Bn * Hkv, cap, HEAD_DIM), dtype=torch.float16, device=dev)
    qf = torch.randn((Bn * Hkv, GQ, HEAD_DIM), dtype=torch.float16, device=dev)

    def fp16_attn():
        s = torch.matmul(qf, kT).float() * scale
        torch.matmul(torch.softmax(s, dim=-1).half(), vf)

    fp16_us = timed(fp16_attn)
    del kT, vf, qf
    if rq:
        # LDS bytes per token and key/value head: the key codeword halves of
        # every stage (M x 256 B, gathered as 16-byte pieces), the weight's
        # float32 adds into M stage bins per query head, and the share of the
        # stage-pair table copies (M x 64 KiB per chunk of tokens)
        chunk = 2 * 8 * (32 // GQ) * 32
        lds_per = M * 256 + M * GQ * 4 + M * 65536 // chunk
        desc = (f"0.75-bit K/V (d=128 K=256 M={M}, one subspace per head; the paper's "
                f"decoding-latency setting)")
    else:
        lds_per = 1024
        desc = "1-bit K/V (d=8 K=256 M=1)"
    return {"decode_attention": {
        "shape": f"{Bn} seq x {cap} tok, {Hq} q / {Hkv} kv heads x {HEAD_DIM}, {desc}, "
                 f"RoPE base 500000",
        "call_us": call_us, "kernel_us": kern_us,
        # a layer's codebooks are fixed across decoding steps: with the
        # tables kept in the workspace (GSRQ_ATTN_TABLES_READY)
        "call_us_tables_ready": ready_us,
        "token_heads_per_s": tok_heads / (call_us * 1e-6),
        "algorithmic_bytes": alg_bytes,
        # LDS bytes: 1-bit layout, 16 key and 16 value codewords gathered
        # (16 B each), the value codewords stored to and read back from the
        # tile: 1 KiB per token and key/value head; 0.75-bit layout above
        "lds_bytes": tok_heads * lds_per,
        "hbm_GBps": alg_bytes / (kern_us * 1e-6) / 1e9,
        "hbm_frac": alg_bytes / (kern_us * 1e-6) / 1e9 / PEAK_HBM_GBPS,
        "fp16_attention_us": fp16_us,
        "speedup_vs_fp16_attention": fp16_us / call_us}}


def attention_cpu_baseline(shape=ATTN_SHAPE, budget_s=10.0, layout="1bit"):
    """Time the float64 oracle on whole sequences of the attention workload
    (unpack, dequantise, RoPE, attention), as many as fit in about budget_s
    seconds (at least one), and scale to token-heads/s of the workload."""
    import numpy as np

    import synth
    from oracle import gsrq_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    Bn, cap, Hkv, GQ = shape["B"], shape["cap"], shape["Hkv"], shape["GQ"]
    rq = layout == "075bit"
    if rq:
        M = ATTN_RQ_STAGES
        case = synth.attn_case_rq(Bn, cap, [cap] * Bn, Hkv, GQ, M=M, seed=0, q_dtype="float16")
        G, d = Hkv, HEAD_DIM
    else:
        M = 1
        case = synth.attn_case(Bn, cap, [cap] * Bn, Hkv, GQ, seed=0, q_dtype="float16")
        G, d = Hkv * HEAD_DIM // 8, 8
    done, t = 0, 0.0
    while done < Bn and (done == 0 or t < budget_s):
        t0 = time.perf_counter()
        kc = O.unpack_codes(case["k_codes"][done], M, G, 256)
        vc = O.unpack_codes(case["v_codes"][done], M, G, 256)
        if rq:
            # keys: the float16 decode of each stage codeword, summed; values:
            # the float32 codewords summed (the inputs the kernel declares)
            kt = (case["k_gain"][..., None] * case["k_shape"]).astype(np.float32)
            vt = (case["v_gain"][..., None] * case["v_shape"]).astype(np.float32)
            kt = kt.astype(np.float16).astype(np.float64)
            k = np.zeros((cap, G, d))
            v = np.zeros((cap, G, d))
            for m in range(M):
                k += kt[m][np.arange(G)[None, :], kc[:, m, :]]
                v += vt[m][np.arange(G)[None, :], vc[:, m, :]].astype(np.float64)
        else:
            k = O.gsrq_decode(kc, case["k_gain"], case["k_shape"])
            v = O.gsrq_decode(vc, case["v_gain"], case["v_shape"])
            k = k.astype(np.float32).astype(np.float16).reshape(cap, Hkv, HEAD_DIM)
            v = v.astype(np.float32).astype(np.float16).reshape(cap, Hkv, HEAD_DIM)
        O.attn_decode(case["q"][done], k, v, 500000.0)
        t += time.perf_counter() - t0
        done += 1
    return {"value": done * cap * Hkv / t, "unit": "token-heads/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"float64 oracle (unpack, decode, float16 rounding, RoPE, attention) on "
                       f"{done} of {Bn} sequences of {cap} tokens x {Hkv} key/value heads "
                       f"({t:.1f} s)")}


def copy_reference(mib, dev):
    """A plain device-to-device copy of mib MiB: the reference dispatch that
    scales the FETCH_SIZE / WRITE_SIZE counters of a profiling run."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    return n * 4


def breakdown(B, step):
    """Per-kernel event times of one extra step (every kind recorded)."""
    import torch
    B.timing_enable(True)
    step()
    torch.cuda.synchronize()
    tim = B.timing_read()
    B.timing_enable(False)
    return tim


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); this path runs on a "
              f"single MI355X and has no multi-GPU mode", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    from paper_2607_01065_amd import gsrq as B

    B.load_library()
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.workload in ("decode_attention_1bit", "decode_attention_075bit"):
        rq = args.workload == "decode_attention_075bit"
        r = attention_measure(B, torch.device("cuda", 0), reps=args.steps,
                              layout="075bit" if rq else "1bit")["decode_attention"]
        line = {"metric": "decode attention token-heads/s over "
                          + ("0.75-bit" if rq else "1-bit") + " coded K/V",
                "value": r["token_heads_per_s"], "unit": "token-heads/s",
                "n_gpus": 1, "steps": args.steps, "warmup": 1,
                "ms_per_step": r["call_us"] / 1e3, "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": "f16",
                "data": "synthetic",
                "config": {"workload": args.workload, "shape": r["shape"]},
                **{k: v for k, v in r.items() if k != "shape"}}
        gbps = r["algorithmic_bytes"] / (r["kernel_us"] * 1e-6) / 1e9
        lds_tbps = r["lds_bytes"] / (r["kernel_us"] * 1e-6) / 1e12
        import hashlib
        tr = TRAFFIC.get(args.workload)
        traffic = None
        if tr is not None:
            src = os.path.join(ROOT, "paper_2607_01065_amd", "csrc", tr["source"])
            sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
            traffic = tr["bytes_per_launch"] if sha == tr["source_sha256_prefix"] else None
        note = ("key codeword pieces of every stage (M x 256 B), float32 weight adds into "
                "M stage bins per query head, stage-pair table copies: per token and "
                "key/value head; peak = 256 CU x 128 B/clk x 2.4 GHz" if rq else
                "codeword gathers, value-tile stores and transposing loads: 1 KiB per token "
                "and key/value head; peak = 256 CU x 128 B/clk x 2.4 GHz; the kernel is bound "
                "by LDS bank conflicts of the random gathers, not by HBM")
        line["roofline"] = {
            "kernel": ("attn_rq_chunk_kernel (unpack + stage-pair dequantise + RoPE + scores + "
                       "softmax + per-codeword value weights)" if rq else
                       "attn_chunk_kernel (unpack + dequantise + RoPE + attention)"),
            "bound": "hbm", "achieved": gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": gbps / PEAK_HBM_GBPS,
            "traffic": traffic, "traffic_unit": "HBM bytes per launch",
            "bytes_per_launch": r["algorithmic_bytes"], "avg_launch_us": r["kernel_us"],
            "lds_view": {"achieved": lds_tbps, "peak": PEAK_LDS_TBPS, "unit": "TB/s",
                         "frac": lds_tbps / PEAK_LDS_TBPS, "bytes_per_launch": r["lds_bytes"],
                         "note": note}}
        if args.copy_ref_mib > 0:
            line["copy_ref_bytes"] = copy_reference(args.copy_ref_mib, torch.device("cuda", 0))
        if not args.no_cpu_baseline:
            line["cpu_baseline"] = attention_cpu_baseline(layout="075bit" if rq else "1bit")
        print(json.dumps(line), flush=True)
        return
    wl = synth.WORKLOADS[args.workload]
    if args.stages > 0:
        import dataclasses
        wl = dataclasses.replace(wl, M=args.stages)
    if wl.layers > 1:
        return full_cache(args, wl)
    N, D, d, K, T, M = wl.N, wl.D, wl.d, wl.K, wl.T, wl.M
    G = D // d
    kv = synth.make_kv(wl, layer=0, seed=0)
    dev = torch.device("cuda", 0)
    caches = []
    for name, X, w, seeds in (("K", kv.keys, kv.w_keys, kv.seeds_keys),
                              ("V", kv.values, kv.w_values, kv.seeds_values)):
        caches.append(dict(
            name=name, X=torch.from_numpy(X).to(dev), w=torch.from_numpy(w).to(dev),
            seeds=[np.ascontiguousarray(seeds[m], dtype=np.int32) for m in range(M)],
            gain=torch.empty((M, G, K), dtype=torch.float32, device=dev),
            shape=torch.empty((M, G, K, d), dtype=torch.float32, device=dev),
            assign=torch.empty((G, N), dtype=torch.int16, device=dev),
            codes=torch.empty((N, B.code_words(N, D, d, K, M)), dtype=torch.int32, device=dev),
            xhat=torch.empty((N, D), dtype=torch.float16, device=dev),
        ))
    # stage inputs after the first: float32 residuals (ping-pong)
    rbuf = [torch.empty((N, D), dtype=torch.float32, device=dev) for _ in range(min(M - 1, 2))]
    ws_train = torch.empty(B.train_workspace_bytes(N, D, d, K), dtype=torch.uint8, device=dev)
    ws_enc = torch.empty(B.encode_workspace_bytes(N, D, d, K, M), dtype=torch.uint8, device=dev)
    iters = []

    def step():
        for c in caches:
            R = c["X"]
            for m in range(M):
                r = B.train_stage(R, d, K, T, seed_rows=c["seeds"][m], w=c["w"],
                                  gain=c["gain"][m], shape=c["shape"][m], assign=c["assign"],
                                  trace=False, workspace=ws_train,
                                  residual=rbuf[m % 2] if m + 1 < M else False)
                iters.append(r.iters)
                R = r.residual
            B.encode(c["X"], c["gain"], c["shape"], codes=c["codes"], workspace=ws_enc)
            B.decode(c["codes"], c["gain"], c["shape"], D, out=c["xhat"])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    iters.clear()
    # events only around the dominant kernel's launches, and only in the
    # first timed step (each event record between dependent kernels costs
    # the GPU a few microseconds); the per-kernel breakdown of the other
    # kernels comes from one instrumented step afterwards
    B.timing_enable(True, kinds=["assign"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step()
        if k == 0:
            B.timing_enable(False)   # records of the enqueued launches are kept
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    tim_timed = B.timing_read()
    n_iters = len(iters)
    tim = breakdown(B, step)
    del iters[n_iters:]
    tim["assign"] = tim_timed["assign"]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    vectors = 2 * N * (D // HEAD_DIM)
    value = vectors / (ms_per_step / 1e3)

    def avg_us(kind):
        ms, n = tim[kind]
        return (ms / n * 1e3) if n else None

    a_us, f_us, e_us, dcd_us = avg_us("assign"), avg_us("finalize"), avg_us("encode"), avg_us("decode")
    import hashlib
    traffic = None
    tr = TRAFFIC.get(wl.name)
    if tr is not None:
        src = os.path.join(ROOT, "paper_2607_01065_amd", "csrc", tr["source"])
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        traffic = tr["bytes_per_launch"] if sha == tr["source_sha256_prefix"] else None
    iters_run = float(torch.stack(iters).float().mean().item()) if iters else float("nan")
    flops_assign = 2.0 * N * D * K                         # eq. (5) scores, one pass
    achieved = flops_assign / (a_us * 1e-6) / 1e12
    dec_bytes = N * M * G * np.log2(K) / 8 + N * D * 2     # packed codes in, fp16 out
    out = {
        "metric": METRIC, "value": value, "unit": "vectors/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "shape": wl.note, "tokens": N, "kv_heads": D // HEAD_DIM,
                   "head_dim": HEAD_DIM, "d": d, "K": K, "M": M, "T": T, "caches": "K and V",
                   "bits_per_element": B.bits_per_element(d, K, M)},
        "encode_vectors_per_s": 2 * N * (D // HEAD_DIM) / (e_us * 1e-6 * tim["encode"][1]),
        "gskm_iter_per_s": 1e6 / (a_us + (f_us or 0.0) + (avg_us("accumulate") or 0.0)
                                  + (avg_us("fragments") or 0.0)),
        "gskm_iters_run_mean": iters_run,
        "decode_GBps": dec_bytes / (dcd_us * 1e-6) / 1e9,
        "decode_hbm_frac": dec_bytes / (dcd_us * 1e-6) / 1e9 / PEAK_HBM_GBPS,
        "kernels_us": {k: {"avg_us": avg_us(k), "launches": tim[k][1]} for k in tim},
        "kernels_us_source": "assign: HIP events around its launches in the first timed "
                             "step; others: one instrumented step after the timed region",
        "roofline": {"kernel": ("assign_accumulate (eq. 5 scores + argmin + weighted sums)"
                               if d <= 8 and K <= 256 else
                               "w_score (eq. 5 scores + argmin; training pass)"),
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_MFMA_F16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_MFMA_F16_TFLOPS,
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch",
                     "flops_per_launch": flops_assign, "avg_launch_us": a_us,
                     "alu_view": {"bound": "alu", "unit": "Tscore/s",
                                  "achieved": N * (D // d) * K / (a_us * 1e-6) / 1e12,
                                  "peak": 39.3,
                                  "note": "argmin epilogue: one VALU lane-op per score is the "
                                          "floor; peak = 256 CU x 64 lanes x 2.4 GHz"}},
    }
    if not args.no_extra:
        out.update(extra_paths(B, caches[0], wl, dev))
    if args.copy_ref_mib > 0:
        out["copy_ref_bytes"] = copy_reference(args.copy_ref_mib, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(kv, wl, min(args.cpu_groups, wl.G))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
