"""Benchmark of the FOCUS hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1]

One step = one pass of the whole prefill hot path over a 1 Mb sequence
(1 000 windows of 1 000 nt, a summary token every 100 nt, 32 heads x 128, bf16):
focus_layout, then focus_compact_kv over every window (10 000 retained rows),
then focus_window_attn over every window in one masked-parallel launch.
Inputs (Q, K, V) are resident in HBM before timing starts.  `value` is input
nucleotides per second over the timed steps.

Also reported on the same JSON line:
  roofline      the attention kernel against the bf16 MFMA peak, timed with
                HIP events on the stream it runs on; `traffic` from the
                committed rocprofv3 counter summary when it matches the current
                kernel source, else null
  cpu_baseline  the float64 oracle on a bounded sample of the same workload
                (whole windows, all heads), extrapolated by visible pairs
  secondary     compaction and decode (batch 16 at ~1 Mb) HBM rates, the dense
                32 kb causal point, streaming (one window per call) prefill, and
                the same 1 Mb prefill under the k-mer-local mask (HBM-bound), the
                fidelity metrics over 1 M positions (HBM-bound), the FOCUS
                adapter update of the summary tokens at 1 Mb (d_model 4096), and
                the fused Q/K/V projection + RoPE + cache write at 1 Mb; as
                context, what plain PyTorch ops reach on the same chip (HBM
                read / write / copy, and a bf16 torch.matmul on the matrix
                cores)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "window-attention tokens/s at 1 Mb context; % MFMA peak (prefill), % HBM BW (decode)"
PEAK_BF16_FLOPS = 2.5e15      # MI355X dense bf16 MFMA
PEAK_HBM = 8.0e12             # MI355X HBM3E bytes/s
# fp32 VALU issue without packed math: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
# lane-instructions/s (a wave64 instruction takes 4 cycles of a SIMD; exp2,
# log2 and sqrt take 8, measured, so they count as two)
PEAK_VALU = 256 * 4 * 16 * 2.4e9
# VALU work per (p, q) element pair of the fidelity metrics from logits, in
# those units: per side max, shift-scale, exp2 (2), sum = 5; square roots of
# the probabilities and the probabilities = 4; L1 2, L2 1, Hellinger 2; log2 p
# and log2 q 2; KL 2; JS: exp2 (2), fma, log2 (2), max, add, sum, 2 fma = 10
FID_VALU_PER_PAIR = 2 * 5 + 4 + 2 + 1 + 2 + 2 + 2 + 10
ATTN_SOURCES = ["paper_2511_14694_amd/csrc/window_attn.hip", "paper_2511_14694_amd/csrc/common.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_window_attn_prefill_1mb.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_hash(paths):
    """Hash of the code of the given sources: comments and whitespace are
    dropped, so editing a comment does not retire counters taken on the same
    code."""
    import re
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p)) as f:
            t = f.read()
        t = re.sub(r"/\*.*?\*/", " ", t, flags=re.S)
        t = re.sub(r"//[^\n]*", "", t)
        h.update(" ".join(t.split()).encode())
    return h.hexdigest()[:16]


def visible_pairs(win_ntok, win_cache_off):
    """Query-key pairs the C(t) mask admits: every window query sees its C_w
    cache rows and the i + 1 window rows up to itself."""
    T = win_ntok.astype(np.int64)
    C = win_cache_off.astype(np.int64)
    return int((T * C + T * (T + 1) // 2).sum())


def kmer_local_pairs(win_ntok, win_cache_off, win_kmer):
    """Query-key pairs the k-mer-local mask admits, in closed form per window:
    a token at offset p of k-mer g sees p + 1 tokens of its k-mer, the g earlier
    summaries of its window and the carried boundary (when C_w > 0)."""
    T = np.asarray(win_ntok, np.int64)
    bnd = (np.asarray(win_cache_off, np.int64) > 0).astype(np.int64)
    k = np.broadcast_to(np.asarray(win_kmer, np.int64), T.shape)
    dense = T * (T + 1) // 2 + T * bnd                                    # k = 0: one k-mer
    kp = np.maximum(k, 0) + 1
    B = np.where(k > 0, (T + kp - 1) // kp, 1)
    nf = B - 1                                                            # full k-mers
    last = T - nf * kp
    full = nf * kp * (kp + 1) // 2 + kp * (nf * (nf - 1) // 2 + nf * bnd)
    tail = last * (last + 1) // 2 + last * (nf + bnd)
    return int(np.where(k > 0, full + tail, dense).sum())


class Timer:
    """HIP events on the current stream (the one every library call uses)."""

    def __init__(self, torch):
        self.torch = torch
        self.marks = {}

    def span(self, name):
        torch = self.torch
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        self.marks.setdefault(name, []).append((s, e))
        return s, e

    def mean_ms(self, name):
        xs = [s.elapsed_time(e) for s, e in self.marks.get(name, [])]
        return float(np.mean(xs)) if xs else float("nan")


class ClockSampler:
    """Samples the GPU's graphics clock (mean over its XCDs, MHz) and socket
    power (W) every few ms while the timed steps run, through amdsmi's GPU
    metrics; reports nothing when amdsmi is unavailable."""

    def __init__(self, period_s=0.005):
        import threading
        self.period = period_s
        self.samples = []
        self.error = None
        self.ok = False
        self._stop = threading.Event()
        self._thread = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[0]
            self.ok = True
        except Exception as e:
            self.ok = False
            self.error = repr(e)

    def _read(self):
        m = self._smi.amdsmi_get_gpu_metrics_info(self._h)
        clks = [c for c in m.get("current_gfxclks", []) if isinstance(c, (int, float)) and c < 0xFFFF]
        clk = float(np.mean(clks)) if clks else float(m.get("current_gfxclk", float("nan")))
        pw = m.get("current_socket_power", float("nan"))
        return clk, float(pw) if isinstance(pw, (int, float)) else float("nan")

    def __enter__(self):
        import threading
        if self.ok:
            def loop():
                while not self._stop.is_set():
                    try:
                        self.samples.append(self._read())
                    except Exception as e:
                        self.error = repr(e)
                    time.sleep(self.period)
            self._thread = threading.Thread(target=loop, daemon=True)
            self._thread.start()
        return self

    def __exit__(self, *a):
        self._stop.set()
        if self._thread:
            self._thread.join()
        return False

    def summary(self):
        # samples taken while the clock is up (the GPU busy: above 1 GHz; the
        # idle clock reads ~0.5 GHz, e.g. between launches), not idle ones
        busy = [c for c in self.samples if c[0] > 1000]
        if not self.ok or not busy:
            return {"unavailable": self.error or f"{len(self.samples)} samples, none with the clock up"}
        clk = np.array([c[0] for c in busy])
        pw = np.array([c[1] for c in busy])
        return {"gfxclk_MHz_median": float(np.median(clk)), "gfxclk_MHz_mean": float(clk.mean()),
                "gfxclk_MHz_min": float(clk.min()), "gfxclk_MHz_max": float(clk.max()),
                "socket_power_W_mean": float(np.nanmean(pw)) if np.isfinite(pw).any() else None,
                "samples": len(busy), "samples_idle": len(self.samples) - len(busy),
                "source": "amdsmi GPU metrics (current_gfxclks, current_socket_power)"}


def prefill_setup(torch, F, fw, w):
    dev = torch.device("cuda:0")
    seq = [w.seq_nt] * w.batch
    kmer = fw.kmer_draw(w)
    totals = F.focus_layout_plan(seq, w.window_nt, kmer)
    seq_d = torch.as_tensor(np.asarray(seq, np.int64), device=dev)
    kmer_d = torch.as_tensor(kmer, device=dev)
    lay = F.focus_layout(totals, seq_d, w.window_nt, kmer_d, device=dev)
    n = totals.n_tokens
    q, k, v = fw.qkv(n, w, device=dev)
    cap = max(totals.max_cache_per_seq, 1)
    td = q.dtype
    ck = torch.empty(w.batch, cap, w.kv_heads, w.head_dim, dtype=td, device=dev)
    cv = torch.empty_like(ck)
    clen = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(n, w.heads, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    return dict(seq_d=seq_d, kmer_d=kmer_d, totals=totals, lay=lay, q=q, k=k, v=v, ck=ck, cv=cv,
                clen=clen, o=o, lse=lse, w=w)


def prefill_step(torch, F, s, timer=None):
    w = s["w"]
    t = timer.span if timer else None
    if t:
        a = t("layout")
        a[0].record()
    F.focus_layout(s["totals"], s["seq_d"], w.window_nt, s["kmer_d"], out=s["lay"])
    if t:
        a[1].record()
        a = t("compact")
        a[0].record()
    s["clen"].zero_()
    F.focus_compact_kv(s["lay"], s["k"], s["v"], s["ck"], s["cv"], s["clen"])
    if t:
        a[1].record()
        a = t("attn")
        a[0].record()
    F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"])
    if t:
        a[1].record()


def kv_bytes(w, totals):
    """Retained summary K/V against the K/V a dense decoder keeps for the same
    bases, per attention layer, all sequences (the memory the paper's scaling
    curves measure; eq. kv-budget / kv-ratio)."""
    elt = 2 if w.dtype == "bf16" else 4
    row = 2 * w.kv_heads * w.head_dim * elt            # K and V of one token
    summary = totals.n_summaries * row
    dense = w.seq_nt * w.batch * row
    return {"summary_kv_bytes": summary, "dense_kv_bytes": dense, "ratio": summary / dense}


def secondary_prefill_config(torch, F, fw, name, reps=5):
    """Another prefill configuration, attention only: masked-parallel (every
    window of every sequence in one launch) and streaming (window j of every
    sequence in one call, j = 0, 1, ...), against the bf16 MFMA peak with the
    visible pairs of the drawn layout; plus the summary-KV / dense-KV bytes."""
    w = fw.WORKLOADS[name]
    s = prefill_setup(torch, F, fw, w)
    prefill_step(torch, F, s)          # layout + compaction fill the cache
    timer = Timer(torch)
    for _ in range(reps):
        a = timer.span("mp")
        a[0].record()
        F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"])
        a[1].record()
    torch.cuda.synchronize()
    ms = timer.mean_ms("mp")
    lay = s["lay"]
    pairs = visible_pairs(lay["win_ntok"].cpu().numpy(), lay["win_cache_off"].cpu().numpy())
    flops = 4 * w.head_dim * w.heads * pairs
    # streaming: every sequence's window j per call (the batch advances in step)
    nw = fw.windows_per_seq(w.seq_nt, w.window_nt)
    cu = lay["cu_windows"].cpu().numpy()
    ids = [torch.tensor([int(cu[b]) + j for b in range(w.batch) if int(cu[b]) + j < int(cu[b + 1])],
                        dtype=torch.int32, device="cuda:0") for j in range(nw)]
    n_ws = max(F.focus_window_attn_workspace(lay, s["q"], s["k"], s["v"], s["ck"], s["cv"], i) for i in ids)
    ws = torch.empty(max(n_ws, 16), dtype=torch.uint8, device="cuda:0")

    def stream_pass():
        for i in ids:
            F.focus_window_attn(lay, s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"],
                                win_ids=i, workspace=ws)

    stream_pass()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    stream_pass()
    e1.record()
    torch.cuda.synchronize()
    ms_stream = e0.elapsed_time(e1)
    nt = w.seq_nt * w.batch
    out = {"workload": f"{w.name}: batch {w.batch} x {w.seq_nt:,} nt, windows of {w.window_nt} nt, "
                       + (f"one summary per {w.kmer} nt" if w.kmer else
                          f"cadence per window drawn from {list(w.kmer_choices)}")
                       + f", {w.heads} x {w.head_dim} {w.dtype}",
           "visible_pairs_per_head": pairs, "flops": flops,
           "masked_parallel": {"ms": ms, "nt_per_s": nt / (ms * 1e-3), "tflops": flops / ms / 1e9,
                               "frac_mfma": flops / (ms * 1e-3) / PEAK_BF16_FLOPS},
           "streaming": {"calls": nw, "windows_per_call": w.batch, "ms": ms_stream,
                         "nt_per_s": nt / (ms_stream * 1e-3), "frac_mfma": flops / (ms_stream * 1e-3) / PEAK_BF16_FLOPS,
                         "workspace_bytes": n_ws},
           "kv_bytes_per_layer": kv_bytes(w, s["totals"])}
    del s, ws
    torch.cuda.empty_cache()
    return out


def cpu_baseline_decode(budget_s=12.0):
    """The decode oracle as it stands on the batch-16 ~1 Mb decode workload:
    for every sequence, the states at steps 1, 2, 3, the first summary step,
    the first window end and the last step (lengths from the oracle's own
    replay of the layout rule, random K/V rows of those lengths), one oracle
    step's attention each, until the time budget is used; the 1000-step run is
    extrapolated by the keys read."""
    import focus_workloads as fw
    from oracle.decode import DecodeSequence
    w = fw.WORKLOADS["decode_b16_1mb"]
    W, k, steps, H, Hkv, D = w.window_nt, w.kmer, w.decode_steps, w.heads, w.kv_heads, w.head_dim
    starts = fw.decode_positions(w)
    rng = np.random.default_rng(fw.BASE_SEED)
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:
        limiter = None
    samples, total_keys = [], 0
    z = np.zeros((1, 1), np.float32)
    for b in range(w.batch):
        nb, ns, ok = DecodeSequence.replay_counters(W, k, int(starts[b]))
        st = DecodeSequence(W, k, [z] * (w.decode_cache_rows + ns), [z] * (w.decode_cache_rows + ns),
                            [z] * nb, [z] * nb, nb, ok)
        lens, first_s, first_e = [], None, None
        for i in range(steps):
            _, _, kind, end = st.step(None, z, z, compute=False)
            lens.append((st.cache_len, st.win_len if not end else st.win_len))
            if kind == 1 and first_s is None:
                first_s = i
            if end and first_e is None:
                first_e = i
        # keys the step attends over: the lengths right after its append
        keys = [c + wl for c, wl in lens]
        total_keys += sum(keys)
        for i in sorted({0, 1, 2, first_s or 0, first_e or 0, steps - 1}):
            samples.append((b, i, keys[i]))
    done_keys, t = 0, 0.0
    nmax = max(nk for _, _, nk in samples)
    pool_k = rng.standard_normal((nmax, Hkv, D)).astype(np.float32)
    pool_v = rng.standard_normal((nmax, Hkv, D)).astype(np.float32)
    for b, i, nk in samples:
        st = DecodeSequence(W, k, list(pool_k[:nk]), list(pool_v[:nk]), [], [], 0, 0)
        q = rng.standard_normal((H, D))
        c0 = time.perf_counter()
        st.attend(q)
        t += time.perf_counter() - c0
        done_keys += nk
        if t > budget_s:
            break
    if limiter is not None:
        limiter.restore_original_limits()
    t_full = t * total_keys / done_keys
    return {"value": w.batch * steps / t_full, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": (f"oracle decode attention at {len(samples)} sampled (sequence, step) states of "
                       f"decode_b16_1mb (steps 1, 2, 3, first summary, first window end, {steps}), "
                       f"{done_keys:,} of {total_keys:,} keys in {t:.1f} s; the {steps}-step run "
                       f"extrapolated by keys to {t_full:.0f} s")}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(torch, s, budget_s=20.0):
    """The oracle, as it is, on whole windows of the same workload (all heads):
    the last window first, then earlier ones, until the time budget is used.
    The full-workload time is extrapolated by the visible-pair ratio."""
    from oracle import attention as A
    from oracle.layout import build_layout
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)     # BLAS threads = the host cores this process may use
    except Exception:
        limiter = None
    w = s["w"]
    t_layout0 = time.perf_counter()
    ref = build_layout([w.seq_nt] * w.batch, w.window_nt, fw_kmer(w))
    t_layout = time.perf_counter() - t_layout0
    nw = ref["n_windows"]
    order = [nw - 1, nw // 2, nw // 4, 3 * nw // 4, 1]
    stride = next(p for p in (379, 383, 389, 397) if nw % p)   # co-prime: visits every window
    order += [i for i in ((j * stride) % nw for j in range(nw)) if i not in order]
    done, pairs, t_attn = [], 0, 0.0
    for wi in order:
        t0, T = int(ref["win_tok_off"][wi]), int(ref["win_ntok"][wi])
        idx = A.cache_token_indices(ref, wi)
        f64 = lambda x: x.float().cpu().numpy().astype(np.float64)  # noqa: E731
        q, k, v = f64(s["q"][t0:t0 + T]), f64(s["k"][t0:t0 + T]), f64(s["v"][t0:t0 + T])
        ti = torch.as_tensor(idx, device=s["k"].device)
        ck, cv = f64(s["k"][ti]), f64(s["v"][ti])
        c0 = time.perf_counter()
        A.window_attention(q, k, v, ck, cv)
        t_attn += time.perf_counter() - c0
        done.append(wi)
        pairs += T * len(idx) + T * (T + 1) // 2
        if t_attn > budget_s:
            break
    total_pairs = visible_pairs(ref["win_ntok"], ref["win_cache_off"])
    t_full = t_attn * total_pairs / pairs + t_layout
    if limiter is not None:
        limiter.restore_original_limits()
    return {"value": w.seq_nt * w.batch / t_full, "unit": "nt/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": (f"oracle window attention on {len(done)} windows {_span(done)} (all {w.heads} heads, "
                       f"{pairs:,} of {total_pairs:,} visible pairs per head) in {t_attn:.1f} s, "
                       f"plus the full oracle layout walk ({t_layout:.1f} s); full-workload time "
                       f"extrapolated by the visible-pair ratio to {t_full:.0f} s")}


def _span(ids, show=6):
    return str(ids) if len(ids) <= show else "[" + ", ".join(map(str, ids[:show])) + ", ...]"


def fw_kmer(w):
    import focus_workloads as fw
    return fw.kmer_draw(w)


def traffic_entry():
    if not os.path.exists(TRAFFIC_FILE):
        return None
    rec = json.load(open(TRAFFIC_FILE))
    if rec.get("source_hash") != source_hash(ATTN_SOURCES):
        return None
    return rec.get("bytes_per_launch")


def secondary_compaction(torch, F, s, timer, reps=10):
    """Bulk compaction at 1 Mb with the 256 MB last-level cache flushed first."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda:0")
    for _ in range(reps):
        flush.fill_(1)
        a = timer.span("compact_cold")
        a[0].record()
        F.focus_compact_kv(s["lay"], s["k"], s["v"], s["ck"], s["cv"], s["clen"])
        a[1].record()
    torch.cuda.synchronize()
    w = s["w"]
    row = w.kv_heads * w.head_dim * 2
    nbytes = s["totals"].n_summaries * row * 2 * 2          # K and V, read + write
    ms = timer.mean_ms("compact_cold")
    return {"rows": s["totals"].n_summaries, "bytes": nbytes, "ms": ms,
            "GBps": nbytes / ms / 1e6, "frac_hbm": nbytes / (ms * 1e-3) / PEAK_HBM}


def secondary_hbm_reference(torch, nbytes=4 << 30, reps=10):
    """What plain PyTorch device ops reach on this machine's HBM (context for the
    HBM-bound kernels' fractions; not part of the hot path): a row-wise max
    over 4 GiB (read), a fill (write) and a copy (read + write)."""
    x = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").normal_()
    y = torch.empty_like(x)

    def t(f):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    read = nbytes / (t(lambda: torch.amax(x.view(-1, 4096), dim=1)) * 1e-3)
    write = nbytes / (t(lambda: y.fill_(1.0)) * 1e-3)
    copy = 2 * nbytes / (t(lambda: y.copy_(x)) * 1e-3)
    del x, y
    torch.cuda.empty_cache()
    return {"read_GBps": read / 1e9, "write_GBps": write / 1e9, "copy_GBps": copy / 1e9,
            "note": "torch.amax over rows (read), fill_ (write), copy_ (read + write) of 4 GiB"}


def secondary_mfma_reference(torch, m=262144, n=4096, k=4096, reps=10):
    """What the vendor GEMM (torch.matmul on bf16, hipBLASLt) reaches on this
    box's matrix cores under the same power limit (context for the MFMA-bound
    kernels' fractions; not part of the hot path)."""
    a = torch.empty(m, k, dtype=torch.bfloat16, device="cuda:0").normal_()
    b = (torch.empty(k, n, device="cuda:0").normal_() / 64).to(torch.bfloat16)
    c = torch.empty(m, n, dtype=torch.bfloat16, device="cuda:0")
    torch.matmul(a, b, out=c)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        torch.matmul(a, b, out=c)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b, c
    torch.cuda.empty_cache()
    tf = 2.0 * m * n * k / (ms * 1e-3) / 1e12
    return {"gemm": f"{m} x {n} x {k} bf16 (torch.matmul)", "ms": ms, "tflops": tf,
            "frac_mfma": tf * 1e12 / PEAK_BF16_FLOPS}


def secondary_decode(torch, F, fw, steps=None):
    """Batch-16 decode at ~1 Mb: 10 000 cached summaries plus a partial window.
    A step is the device schedule (the next token's kind) + focus_decode_step."""
    w = fw.WORKLOADS["decode_b16_1mb"]
    dev = torch.device("cuda:0")
    steps = steps or w.decode_steps
    B, H, Hkv, D = w.batch, w.heads, w.kv_heads, w.head_dim
    starts = fw.decode_positions(w)
    sched = F.DecodeSchedule(B, w.window_nt, None, w.kmer, device=dev)
    n_sum0 = sched.start(starts).clone()
    sched0 = [t.clone() for t in (sched.win_index, sched.bases_in_window, sched.bases_in_kmer)]
    cap_c = w.decode_cache_rows + 2 * (-(-w.window_nt // w.kmer)) + 8
    seed = fw.seed_for(w.index, "cache_k")
    cache_k = fw.randn((B, cap_c, Hkv, D), w.dtype, seed + 1, dev)
    cache_v = fw.randn((B, cap_c, Hkv, D), w.dtype, seed + 2, dev)
    win_k = fw.randn((B, w.window_nt, Hkv, D), w.dtype, seed + 3, dev)
    win_v = fw.randn((B, w.window_nt, Hkv, D), w.dtype, seed + 4, dev)
    sq = fw.randn((steps, B, H, D), w.dtype, seed + 5, dev)
    sk = fw.randn((steps, B, Hkv, D), w.dtype, seed + 6, dev)
    sv = fw.randn((steps, B, Hkv, D), w.dtype, seed + 7, dev)
    cache_len = (n_sum0 + w.decode_cache_rows).to(torch.int32)
    win_len = sched.bases_in_window.clone()

    def reset_sched():
        for t, t0 in zip((sched.win_index, sched.bases_in_window, sched.bases_in_kmer), sched0):
            t.copy_(t0)

    # the kinds the schedule will give (a dry run), for the algorithmic byte count
    kinds = torch.empty(steps, B, dtype=torch.uint8, device=dev)
    for i in range(steps):
        kinds[i].copy_(sched.next_kind())
    kh = kinds.cpu().numpy()
    cl = cache_len.cpu().numpy().astype(np.int64)
    wl = win_len.cpu().numpy().astype(np.int64)
    keys = 0
    for i in range(steps):
        summ = (kh[i] & 1) > 0
        cl += summ
        wl += ~summ
        keys += int((cl + wl).sum())
        wl[(kh[i] & 2) > 0] = 0
    row = Hkv * D * 2
    nbytes = keys * row * 2 + steps * B * (2 * H * D * 2 + 2 * row + H * 4)
    o = torch.empty(B, H, D, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(B, H, dtype=torch.float32, device=dev)
    ws = torch.empty(F.focus_decode_workspace(sq[0], sk[0], cache_k, win_k), dtype=torch.uint8, device=dev)
    # warm-up on copies of the state, then the timed run from the initial state
    st = [cache_len.clone(), win_len.clone()]
    reset_sched()
    for i in range(min(20, steps)):
        F.focus_decode_step(sq[i], sk[i], sv[i], sched.next_kind(), cache_k, cache_v, st[0], win_k, win_v, st[1],
                            o=o, lse=lse, workspace=ws)
    reset_sched()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        F.focus_decode_step(sq[i], sk[i], sv[i], sched.next_kind(), cache_k, cache_v, cache_len, win_k, win_v,
                            win_len, o=o, lse=lse, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    return {"workload": "decode_b16_1mb: batch 16, 32 x 128 bf16, 10 000 cached summaries + partial window, "
                        f"{steps} steps (each: device schedule + decode step)",
            "tokens_per_s": B * steps / (ms * 1e-3), "ms_per_step": ms / steps,
            "bytes_per_step": nbytes / steps, "GBps": nbytes / ms / 1e6,
            "frac_hbm": nbytes / (ms * 1e-3) / PEAK_HBM}


def secondary_dense(torch, F, fw, reps=3):
    w = fw.WORKLOADS["dense_32kb"]
    s = prefill_setup(torch, F, fw, w)
    F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"])
    timer = Timer(torch)
    for _ in range(reps):
        a = timer.span("dense")
        a[0].record()
        F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"])
        a[1].record()
    torch.cuda.synchronize()
    ms = timer.mean_ms("dense")
    n = w.seq_nt
    flops = 4 * w.head_dim * w.heads * (n * (n + 1) // 2)
    return {"workload": "dense_32kb: one 32 000-token causal window, no summaries, 32 x 128 bf16",
            "ms": ms, "tflops": flops / ms / 1e9, "frac_mfma": flops / (ms * 1e-3) / PEAK_BF16_FLOPS,
            "dense_1mb_extrapolated_s": ms * 1e-3 * (1e6 / n) ** 2}


def secondary_kmer_local(torch, F, fw, s, timer, reps=5):
    """The same 1 Mb layout under the k-mer-local mask (Section 3.2 rule): every
    window in one launch.  Bound by HBM: Q, K, V and O cross it once."""
    mask = F.FOCUS_MASK_KMER_LOCAL
    F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"], mask=mask)
    for _ in range(reps):
        a = timer.span("kmer_local")
        a[0].record()
        F.focus_window_attn(s["lay"], s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"], mask=mask)
        a[1].record()
    torch.cuda.synchronize()
    ms = timer.mean_ms("kmer_local")
    w, tot = s["w"], s["totals"]
    lay = s["lay"]
    pairs = kmer_local_pairs(lay["win_ntok"].cpu().numpy(), lay["win_cache_off"].cpu().numpy(), fw.kmer_draw(w))
    flops = 4 * w.head_dim * w.heads * pairs
    per_tok = w.heads * w.head_dim * 2 * 2 + 2 * w.kv_heads * w.head_dim * 2 + w.heads * 4   # q, o, k, v, lse
    nbytes = tot.n_tokens * per_tok + tot.n_windows * 2 * w.kv_heads * w.head_dim * 2     # + boundary rows
    return {"workload": f"{w.name} under FOCUS_MASK_KMER_LOCAL, all windows in one launch", "ms": ms,
            "nt_per_s": w.seq_nt * w.batch / (ms * 1e-3), "visible_pairs_per_head": pairs,
            "tflops": flops / ms / 1e9, "bytes": nbytes, "GBps": nbytes / ms / 1e6,
            "bound": "hbm", "frac_hbm": nbytes / (ms * 1e-3) / PEAK_HBM}


def secondary_fidelity(torch, F, fw, reps=5):
    """Fidelity metrics (L1, L2, Hellinger, JS, KL per position) over 1 M
    positions, for 4 nucleotides (f32 logits) and a 512-entry vocabulary (bf16
    logits).  Both logit rows are read once and 5 floats written (HBM bound);
    the per-element arithmetic (FID_VALU_PER_PAIR at PEAK_VALU) is the other
    bound, and the larger of the two is the one reported as "bound"."""
    res = {}
    for name, (n, vocab, dtype) in fw.FIDELITY.items():
        p, q = fw.fidelity_logits(n, vocab, dtype, seed=fw.BASE_SEED, device="cuda:0")
        out = torch.empty(n, F.FOCUS_FID_N, dtype=torch.float32, device="cuda:0")
        F.focus_fidelity(p, q, out=out)
        e = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in e:
            a.record()
            F.focus_fidelity(p, q, out=out)
            b.record()
        torch.cuda.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in e) / reps
        nbytes = 2 * n * vocab * p.element_size() + n * F.FOCUS_FID_N * 4
        valu = n * vocab * FID_VALU_PER_PAIR
        t_hbm, t_alu = nbytes / PEAK_HBM, valu / PEAK_VALU
        bound = "alu" if t_alu > t_hbm else "hbm"
        res[name] = {"positions": n, "vocab": vocab, "dtype": dtype, "ms": ms, "bytes": nbytes,
                     "GBps": nbytes / ms / 1e6, "frac_hbm": nbytes / (ms * 1e-3) / PEAK_HBM,
                     "valu_lane_ops": valu, "frac_alu": valu / (ms * 1e-3) / PEAK_VALU,
                     "bound": bound, "frac": max(t_hbm, t_alu) / (ms * 1e-3)}
        del p, q, out
    return res


def secondary_adapter(torch, F, fw, reps=3, d_model=4096):
    """The FOCUS adapter update of the summary tokens (eq. focus-attn) on the
    1 Mb layout with an Evo-2-scale layer (d_model 4096, 32 x 128): W_K / W_V
    over every token, the adapter's retained K/V, W_Q over the summaries, the
    summary-query attention and W_O.  Random weights N(0, 1/d)."""
    w = fw.WORKLOADS["prefill_1mb"]
    H, Hkv, D = w.heads, w.kv_heads, w.head_dim
    seq = [w.seq_nt] * w.batch
    km = fw.kmer_draw(w)
    tot = F.focus_layout_plan(seq, w.window_nt, km)
    lay = F.focus_layout(tot, seq, w.window_nt, km, device="cuda:0")
    hid = fw.randn((tot.n_tokens, d_model), "bf16", fw.BASE_SEED, "cuda:0")
    sc = 1.0 / np.sqrt(d_model)
    wq = (fw.randn((d_model, H * D), "f32", 1, "cuda:0") * sc).to(torch.bfloat16)
    wk = (fw.randn((d_model, Hkv * D), "f32", 2, "cuda:0") * sc).to(torch.bfloat16)
    wv = (fw.randn((d_model, Hkv * D), "f32", 3, "cuda:0") * sc).to(torch.bfloat16)
    wo = (fw.randn((H * D, d_model), "f32", 4, "cuda:0") / np.sqrt(H * D)).to(torch.bfloat16)
    ws = torch.empty(F.focus_adapter_layer_workspace(lay, hid, wq, wk, wv, wo, H, Hkv), dtype=torch.uint8,
                     device="cuda:0")
    out = torch.empty(tot.n_summaries, d_model, dtype=torch.bfloat16, device="cuda:0")
    F.focus_adapter_layer(lay, hid, wq, wk, wv, wo, H, Hkv, out=out, workspace=ws)
    e = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in e:
        a.record()
        F.focus_adapter_layer(lay, hid, wq, wk, wv, wo, H, Hkv, out=out, workspace=ws)
        b.record()
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in e) / reps
    # the attention alone, on the workspace's projections (same launch the layer makes)
    nt, ns = tot.n_tokens, tot.n_summaries
    kv_b = nt * Hkv * D * 2
    k = ws[:kv_b].view(torch.bfloat16).view(nt, Hkv, D)
    off = -(-kv_b // 256) * 256
    v = ws[off:off + kv_b].view(torch.bfloat16).view(nt, Hkv, D)
    qs = torch.empty(ns, H, D, dtype=torch.bfloat16, device="cuda:0")
    F.focus_gemm(hid, wq, out=qs.view(ns, H * D), a_rows=lay["sum_tok"])
    cap = max(tot.max_cache_per_seq, 1)
    ck = torch.empty(w.batch, cap, Hkv, D, dtype=torch.bfloat16, device="cuda:0")
    cv = torch.empty_like(ck)
    F.focus_compact_kv(lay, k, v, ck, cv)
    F.focus_adapter_attn(lay, qs, k, v, ck, cv)
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for _ in range(reps):
        F.focus_adapter_attn(lay, qs, k, v, ck, cv)
    a1.record()
    torch.cuda.synchronize()
    attn_ms = a0.elapsed_time(a1) / reps
    nsum = lay["win_nsum"].cpu().numpy()
    st = lay["sum_tok"].cpu().numpy()
    win_of = np.repeat(np.arange(tot.n_windows), nsum)
    rows = st - lay["win_tok_off"].cpu().numpy()[win_of]
    cache_off = lay["win_cache_off"].cpu().numpy().astype(np.int64)
    pairs = int((cache_off[win_of] + rows + 1).sum())
    attn_flops = 4 * D * H * pairs
    # algorithmic bytes: every K/V row a summary sees, once -- a window's rows
    # up to its last summary's, and each sequence's cache prefix up to its
    # largest C_w -- plus the summary queries read, outputs and LSE written
    last = np.cumsum(nsum) - 1
    win_rows = int((rows[last[nsum > 0]] + 1).sum())
    seq_of = lay["win_seq"].cpu().numpy()
    cache_rows = sum(int(cache_off[seq_of == b].max(initial=0)) for b in range(w.batch))
    attn_bytes = 2 * Hkv * D * 2 * (win_rows + cache_rows) + 2 * ns * H * D * 2 + ns * H * 4
    gemm_flops = 2 * nt * d_model * 2 * Hkv * D + 2 * ns * d_model * H * D * 2
    flops = attn_flops + gemm_flops
    return {"workload": f"prefill_1mb layout, d_model {d_model}, {H} x {D} heads, bf16, random weights",
            "ms": ms, "tflops": flops / ms / 1e9, "frac_mfma": flops / (ms * 1e-3) / PEAK_BF16_FLOPS,
            "gemm_flops": gemm_flops,
            "attention": {"ms": attn_ms, "visible_pairs_per_head": pairs, "bound": "hbm",
                          "algorithmic_bytes": attn_bytes, "gb_per_s": attn_bytes / attn_ms / 1e6,
                          "frac_hbm": attn_bytes / (attn_ms * 1e-3) / PEAK_HBM,
                          "tflops": attn_flops / attn_ms / 1e9,
                          "frac_mfma": attn_flops / (attn_ms * 1e-3) / PEAK_BF16_FLOPS}}


def secondary_qkv_projection(torch, F, fw, reps=3, d_model=4096):
    """The layer's Q/K/V projection at 1 Mb (d_model 4096 -> 32 + 2 x 32 heads
    of 128) with rotary positions at the augmented-stream index and the summary
    K/V written straight into the cache (no separate compaction pass)."""
    w = fw.WORKLOADS["prefill_1mb"]
    H, Hkv, D = w.heads, w.kv_heads, w.head_dim
    seq = [w.seq_nt] * w.batch
    km = fw.kmer_draw(w)
    tot = F.focus_layout_plan(seq, w.window_nt, km)
    lay = F.focus_layout(tot, seq, w.window_nt, km, device="cuda:0")
    hid = fw.randn((tot.n_tokens, d_model), "bf16", fw.BASE_SEED + 1, "cuda:0")
    wqkv = (fw.randn((d_model, (H + 2 * Hkv) * D), "f32", 5, "cuda:0") / np.sqrt(d_model)).to(torch.bfloat16)
    q = torch.empty(tot.n_tokens, H, D, dtype=torch.bfloat16, device="cuda:0")
    k = torch.empty(tot.n_tokens, Hkv, D, dtype=torch.bfloat16, device="cuda:0")
    v = torch.empty_like(k)
    ck = torch.empty(w.batch, max(tot.max_cache_per_seq, 1), Hkv, D, dtype=torch.bfloat16, device="cuda:0")
    cv = torch.empty_like(ck)
    run = lambda: F.focus_qkv_project(lay, hid, wqkv, H, Hkv, 10000.0, q=q, k=k, v=v, cache_k=ck, cache_v=cv)  # noqa
    run()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    flops = 2 * tot.n_tokens * d_model * (H + 2 * Hkv) * D
    return {"workload": f"prefill_1mb layout, d_model {d_model} -> ({H} + 2 x {Hkv}) x {D}, RoPE theta 1e4, "
                        "summary K/V written to the cache in the epilogue",
            "ms": ms, "tflops": flops / ms / 1e9, "frac_mfma": flops / (ms * 1e-3) / PEAK_BF16_FLOPS}


def secondary_streaming(torch, F, s, n_windows=200):
    """Streaming prefill: one window per call (last n_windows windows)."""
    lay = s["lay"]
    nw = lay.totals.n_windows
    ids = [torch.tensor([w_], dtype=torch.int32, device="cuda:0") for w_ in range(nw - n_windows, nw)]
    # key-split scratch (the same size for every single-window launch), allocated once
    n_ws = F.focus_window_attn_workspace(lay, s["q"], s["k"], s["v"], s["ck"], s["cv"], ids[-1])
    split_ws = torch.empty(max(n_ws, 16), dtype=torch.uint8, device="cuda:0")
    no_split = torch.empty(0, dtype=torch.uint8, device="cuda:0")

    def run(ws):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in ids:
            F.focus_window_attn(lay, s["q"], s["k"], s["v"], s["ck"], s["cv"], o=s["o"], lse=s["lse"],
                                win_ids=i, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n_windows

    run(split_ws)
    ms = run(split_ws)
    ms_unsplit = run(no_split)
    return {"windows": n_windows, "ms_per_window": ms, "ms_per_window_unsplit": ms_unsplit,
            "workspace_bytes": n_ws,
            "note": "one launch per window (the last windows, largest caches); keys split over the "
                    "compute units the 128 (head, query tile) items leave idle"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="prefill_1mb")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the FOCUS hot path here runs on a single MI355X and "
              f"has no multi-GPU mode (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    import focus_workloads as fw
    import paper_2511_14694_amd as F
    F._abi.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    w = fw.WORKLOADS[args.workload]
    log(f"setup {w.name}")
    s = prefill_setup(torch, F, fw, w)
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0").fill_(3)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        prefill_step(torch, F, s)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    timer = Timer(torch)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    clock = ClockSampler()
    with clock:
        e0.record()
        for i in range(args.steps):
            prefill_step(torch, F, s, timer)
        e1.record()
        torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    ms_step = total_ms / max(args.steps, 1)
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step")

    lay_np = {k: s["lay"][k].cpu().numpy() for k in ("win_ntok", "win_cache_off")}
    pairs = visible_pairs(lay_np["win_ntok"], lay_np["win_cache_off"])
    flops = 4 * w.head_dim * w.heads * pairs
    attn_ms = timer.mean_ms("attn")
    traffic = traffic_entry()
    nt = w.seq_nt * w.batch
    result = {
        "metric": METRIC,
        "value": nt / (ms_step * 1e-3),
        "unit": "nt/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: batch {w.batch} x {w.seq_nt:,} nt, windows of {w.window_nt} nt, "
                               f"one summary token per {w.kmer} nt, {w.heads} heads x {w.head_dim} "
                               f"{w.dtype}; step = layout + compaction + masked-parallel window attention",
                   "augmented_tokens": s["totals"].n_tokens, "visible_pairs_per_head": pairs},
        "roofline": {"bound": "mfma", "achieved": flops / (attn_ms * 1e-3) / 1e12,
                     "peak": PEAK_BF16_FLOPS / 1e12, "unit": "TFLOP/s",
                     "frac": flops / (attn_ms * 1e-3) / PEAK_BF16_FLOPS, "traffic": traffic,
                     "kernel": "attn_ct<128> (focus_window_attn)", "flops_per_launch": flops,
                     "avg_launch_ms": attn_ms},
        "kernel_ms": {"layout": timer.mean_ms("layout"), "compact": timer.mean_ms("compact"),
                      "attn": attn_ms},
        "augmented_tokens_per_s": s["totals"].n_tokens / (ms_step * 1e-3),
        "clock_under_load": clock.summary(),
        "kv_bytes_per_layer": kv_bytes(w, s["totals"]),
    }
    if not args.no_secondary:
        log("secondary: compaction")
        sec = {"compaction_1mb": secondary_compaction(torch, F, s, timer)}
        log("secondary: HBM reference")
        sec["hbm_reference"] = secondary_hbm_reference(torch)
        log("secondary: MFMA reference")
        sec["mfma_reference"] = secondary_mfma_reference(torch)
        log("secondary: streaming")
        sec["streaming_1mb"] = secondary_streaming(torch, F, s)
        log("secondary: k-mer-local mask")
        sec["kmer_local_1mb"] = secondary_kmer_local(torch, F, fw, s, timer)
        if not args.no_cpu_baseline:
            log("cpu baseline (oracle)")
            result["cpu_baseline"] = cpu_baseline(torch, s, args.cpu_budget)
            log("cpu baseline (decode oracle)")
            result["cpu_baseline"]["decode"] = cpu_baseline_decode()
        del s
        torch.cuda.empty_cache()
        log("secondary: decode")
        sec["decode_b16_1mb"] = secondary_decode(torch, F, fw)
        torch.cuda.empty_cache()
        for name in ("prefill_100kb", "ragged_b8_256kb"):
            log(f"secondary: {name}")
            sec[name] = secondary_prefill_config(torch, F, fw, name)
        log("secondary: dense 32 kb")
        sec["dense_32kb"] = secondary_dense(torch, F, fw)
        torch.cuda.empty_cache()
        log("secondary: fidelity metrics")
        sec["fidelity"] = secondary_fidelity(torch, F, fw)
        torch.cuda.empty_cache()
        log("secondary: FOCUS adapter layer")
        sec["adapter_1mb"] = secondary_adapter(torch, F, fw)
        torch.cuda.empty_cache()
        log("secondary: fused Q/K/V projection")
        sec["qkv_projection_1mb"] = secondary_qkv_projection(torch, F, fw)
        result["secondary"] = sec
    elif not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(torch, s, args.cpu_budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
