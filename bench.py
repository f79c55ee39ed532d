#!/usr/bin/env python3
"""Benchmark of the DeLS-Spec block-drafting hot path on one MI355X.

A step is one pass of the whole path over one batch: dls_draft_block (local head, fusion and
greedy argmax at every draft position, with row statistics) followed by dls_accept_len.  The
default workload is the largest single-GPU drafting configuration: batch 64, block B = 16,
V = 151,936, embedding width 5120, GRU hidden 1024, rank 256, bf16 (Zipf-biased long logits).
Inputs are seeded synthetic tensors already resident in HBM.  Prints one JSON line: the
drafted-token throughput of the step, the roofline of the dominant kernel (the persistent drafting
kernel) with warm and cold per-call timing distributions, and beside them the other launch mode,
the block without statistics, the per-position launches, sampling at T = 1, adaptive fusion and
its pre-pass, the Markov head, prior estimation, the standalone fused combine at the two serving
shapes and every drafting workload; then the CPU oracle timed on the host in fresh subprocesses
(all threads, then 1 thread), which also checks the GPU draft of the timed workload element by
element (the `parity` object).
"""
import argparse
import hashlib
import json
import os
import subprocess
import sys
import tempfile
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
TOL = 2e-2                  # statistics tolerance and near-tie gap of the comparison protocol
STAT_KEYS = ("score", "logprob", "gap", "lse_long", "lse_short", "lse_fused")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------------------------------------
# byte and flop accounting (units: one draft position of the whole batch; a launch drafts B of them)
# ------------------------------------------------------------------------------------------------
def algorithmic_bytes(wl, esize=2):
    """Bytes the method moves per block when every position re-reads the head weights (the
    formulation without weight reuse): per position W_vocab + W_ih + W_hh + W_rank, plus one
    embedding row and one long-logit row per sequence (no prior).  Returns (per block, per step)."""
    V, d, H, r = wl.V, wl.d, wl.H, wl.r
    per_step = (V * r + 3 * H * d + 3 * H * H + r * H) * esize + wl.batch * (d * esize + V * esize)
    return per_step * wl.B, per_step


def compulsory_bytes(wl, esize=2):
    """Bytes the weight-stationary kernel must move at least per block: the operand-ordered W_vocab,
    W_hh and W_rank once, then per position one folded-table row (3H float32) and one long-logit row
    per sequence."""
    V, H, r = wl.V, wl.H, wl.r
    nt = (V + 15) // 16
    once = nt * 16 * r * esize + 3 * H * H * esize + r * H * esize
    return once + wl.B * wl.batch * (3 * H * 4 + V * esize)


def method_flops(wl):
    """Multiply-adds x 2 of one block as the kernels compute it: the vocabulary head, W_hh h and
    W_rank h per position and sequence.  The input projection W_ih E[u] is a table lookup (folded
    once per head), so its flops are not counted."""
    V, H, r = wl.V, wl.H, wl.r
    return 2 * wl.batch * wl.B * (V * r + 3 * H * H + r * H)


KERNEL_SOURCES = ["paper_2607_07409_amd/csrc/draft_persistent.hpp", "paper_2607_07409_amd/csrc/dels_internal.hpp",
                  "paper_2607_07409_amd/csrc/dels_device.hpp", "paper_2607_07409_amd/csrc/build.py"]


def kernel_source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the persistent kernel on `workload` from the committed PMC record, or
    None when there is none or the kernel sources changed after it was taken."""
    path = os.path.join(ROOT, "profiles", f"k_draft_persistent_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as fh:
        for line in fh:
            if line.startswith("#") or ":" not in line:
                continue
            k, v = line.split(":", 1)
            rec[k.strip()] = v.split()[0] if v.split() else ""
    if rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return {k: int(rec[k]) for k in ("traffic_bytes_per_launch", "fetch_bytes_per_launch", "write_bytes_per_launch")
            if k in rec} | ({"dram_read_bytes_per_launch": int(rec["dram_read_bytes_per_launch"])}
                            if "dram_read_bytes_per_launch" in rec else {})


def pct(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs, dtype=np.float64), q))


def dist(us):
    return {"median": round(pct(us, 50), 2), "p10": round(pct(us, 10), 2), "p90": round(pct(us, 90), 2),
            "mean": round(sum(us) / len(us), 2), "calls": len(us)}


def per_call_us(fn, n, torch, scratch=None):
    """Duration of each of n calls of fn (HIP events around each call on the current stream).  With
    `scratch` (a large device buffer) the buffer is overwritten before every call, outside the timed
    events, so that no input of the call is left in the caches (L2, MALL)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    torch.cuda.synchronize()
    for i in range(n):
        if scratch is not None:
            scratch.fill_(i & 0xFF)
        evs[i][0].record()
        fn(i)
        evs[i][1].record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in evs]


def measured_peaks(B, dev, torch, read_gib=4, calls=20):
    """The device's attainable peaks, beside the vendor figures the rooflines are quoted against:
    a read of a read_gib GiB buffer (far larger than L2 and MALL) with 16-byte non-temporal loads
    on every CU, and a bf16 matrix-core loop of 8192 workgroups x 4 waves x 1024 rounds x 4
    independent 32x32x16 products.  Both are checked (the read's checksum words against the buffer's XOR,
    every MFMA lane against its exact value) and timed per call with HIP events; medians."""
    nbytes = read_gib << 30
    buf = torch.empty(nbytes // 4, dtype=torch.int32, device=dev)
    buf.fill_(0x5A5A5A5A)
    buf[-1] = 1  # an odd number of equal words and a 1: the buffer's XOR is 0x5A5A5A5B
    words = B.measure_read(buf)
    read_us = per_call_us(lambda _: B.measure_read(buf, out=words), calls, torch)
    xor = 0
    for w in words.cpu().tolist():
        xor ^= w & 0xFFFFFFFF
    del buf
    torch.cuda.empty_cache()
    groups, iters, x = 8192, 1024, 1.0 / 64
    acc = B.measure_mfma(groups, iters, x, device=dev)
    mfma_us = per_call_us(lambda _: B.measure_mfma(groups, iters, x, out=acc), calls, torch)
    exact = bool((acc == iters * 1024 * x * x).all().item())
    flops = groups * 4 * iters * 4 * 32768
    r_med, m_med = pct(read_us, 50), pct(mfma_us, 50)
    return {"hbm_read_GBs": round(nbytes / (r_med * 1e-6) / 1e9, 1), "hbm_vendor_GBs": HBM_PEAK_GBS,
            "read_bytes": nbytes, "read_us": dist(read_us), "read_checksum_ok": xor == 0x5A5A5A5B,
            "bf16_mfma_TFLOPs": round(flops / (m_med * 1e-6) / 1e12, 1), "bf16_vendor_TFLOPs": BF16_PEAK_TFLOPS,
            "mfma_flops": flops, "mfma_us": dist(mfma_us), "mfma_exact": exact,
            "how": "dls_measure_read over a fresh-filled buffer; dls_measure_mfma (v_mfma_f32_32x32x16_bf16)"}


# ------------------------------------------------------------------------------------------------
# CPU oracle leg: a fresh subprocess per thread count (BLAS threads fixed before numpy loads)
# ------------------------------------------------------------------------------------------------
def oracle_leg(args):
    """Runs in its own process.  Loads the workload the parent saved (the same host inputs the GPU
    drafted from), replays the oracle on sequences of the block with the GPU's tokens forced
    (Algorithm 1 through the plain float64 oracle), times it, and with --oracle-parity compares every
    drafted token and statistic with the oracle's.  Prints one JSON line."""
    import numpy as np
    from oracle import dels_oracle as O
    from paper_2607_07409_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    z = np.load(args.oracle_leg, allow_pickle=False)
    wl = W.WORKLOADS[args.workload]

    class Rows:
        """The embedding rows the replay visits (every other row is never read)."""
        def __init__(self, toks, rows):
            self.m = {int(t): rows[i] for i, t in enumerate(toks)}

        def __getitem__(self, t):
            return self.m[int(t)]

    f32 = lambda k: W.bf16_bits_to_f32(z[k]) if z[k].dtype == np.uint16 else z[k]
    emb = Rows(z["emb_tokens"], f32("emb_rows"))
    head = O.RnnHead(emb, f32("w_ih"), f32("w_hh"), f32("w_rank"), f32("w_vocab"))
    long_h = W.Bf16Array(z["long"]) if z["long"].dtype == np.uint16 else z["long"]
    last, gtok, gst = z["last"], z["tokens"], z["stats"]
    alpha = float(z["alpha"])
    seqs = list(range(wl.batch))
    t0 = time.perf_counter()
    done = []
    ref = None
    for b in seqs:
        r = O.draft_block(head, long_h, last, None, 1.0, alpha, 0.0, force=gtok, sequences=[b])
        if ref is None:
            ref = r
        else:
            for f in ("tokens", "score", "logprob", "gap", "lse_long", "lse_short", "lse_fused", "argmax", "margin"):
                getattr(ref, f)[b] = getattr(r, f)[b]
        done.append(b)
        if not args.oracle_parity and time.perf_counter() - t0 >= args.cpu_seconds:
            break
    el = time.perf_counter() - t0
    out = {"threads": threads, "sequences": len(done), "seconds": el,
           "tokens_per_s": len(done) * wl.B / el}
    if args.oracle_parity:
        near, worst_gap, bad = 0, 0.0, []
        long_f = np.asarray(long_h, dtype=np.float32)
        active = 0
        for b in done:
            for j in range(wl.B):
                active += int(ref.argmax[b, j] != int(np.argmax(long_f[b, j])))
                if ref.argmax[b, j] != gtok[b, j]:
                    if ref.gap[b, j] < TOL and ref.margin[b, j] < TOL:
                        near += 1
                        worst_gap = max(worst_gap, float(ref.gap[b, j]))
                    else:
                        bad.append((b, j))
        errs = {}
        for i, k in enumerate(STAT_KEYS):
            if k == "gap":
                continue
            g = gst[done, :, i].astype(np.float64)
            r = getattr(ref, k)[done].astype(np.float64)
            nan = np.isnan(r)
            errs[k] = float(np.max(np.abs(g[~nan] - r[~nan]))) if (~nan).any() else 0.0
            if not np.array_equal(np.isnan(g), nan):
                errs[k] = float("inf")
        acc_ok = bool(np.array_equal(O.accept_len(gtok, z["targets"]), z["accept"]))
        out["parity"] = {"sequences": len(done), "positions": len(done) * wl.B,
                         "tokens_equal": int(sum(int(ref.argmax[b, j] == gtok[b, j]) for b in done
                                                 for j in range(wl.B))),
                         "near_ties": near, "max_near_tie_gap": worst_gap, "mismatches_outside_tolerance": len(bad),
                         "max_abs_err": errs, "tolerance": TOL, "accept_len_equal": acc_ok,
                         "fusion_active": active / (len(done) * wl.B),
                         "ok": (not bad) and acc_ok and all(e <= TOL for e in errs.values())}
    print(json.dumps(out), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def run_oracle_subprocess(npz, args, threads, parity):
    env = dict(os.environ)
    for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS"):
        env[k] = str(threads)
    env["HIP_VISIBLE_DEVICES"] = ""          # the oracle leg never touches the GPU
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--oracle-leg", npz, "--workload", args.workload,
           "--cpu-seconds", str(args.cpu_seconds)] + (["--oracle-parity"] if parity else [])
    p = subprocess.run(cmd, env=env, capture_output=True, text=True, timeout=900)
    if p.returncode != 0:
        raise RuntimeError(f"oracle leg failed ({p.returncode}):\n{p.stderr[-3000:]}")
    return json.loads(p.stdout.strip().splitlines()[-1])


# ------------------------------------------------------------------------------------------------
# other drafting workloads (timing only: device-generated weights of the stress recipe)
# ------------------------------------------------------------------------------------------------
def time_workload(B, W, wl, dev, torch, n=100):
    """Warm per-call draft-block time of one workload with device-generated weights of the stress
    recipe (E ~ N(0,1), W_ih ~ N(0,1/d), W_hh, W_rank ~ N(0,1/H), W_vocab ~ N(0,100/r)) and long
    logits 3 N(0,1) + 8 on one token per row: the timing needs the shapes and the value scale,
    not the oracle's exact values (parity runs on the seeded generators in the tests)."""
    import math
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    g = torch.Generator(device=dev).manual_seed(1000 + wl.seed)

    def rnd(shape, sd):
        return (torch.randn(shape, generator=g, device=dev, dtype=torch.float32) * sd).to(dt)

    V, d, H, r = wl.V, wl.d, wl.H, wl.r
    head = B.LocalHead(rnd((V, d), 1.0), rnd((3 * H, d), 1 / math.sqrt(d)), rnd((3 * H, H), 1 / math.sqrt(H)),
                       rnd((r, H), 1 / math.sqrt(H)), rnd((V, r), 10 / math.sqrt(r)))
    if wl.dtype == "bf16":
        head.prepare()
    L = rnd((wl.batch, wl.B, V), 3.0)
    hot = torch.randint(0, V, (wl.batch, wl.B, 1), generator=g, device=dev)
    L.scatter_add_(2, hot, torch.full((wl.batch, wl.B, 1), 8.0, device=dev, dtype=dt))
    last = torch.randint(0, V, (wl.batch,), generator=g, device=dev, dtype=torch.int32)
    tok = torch.empty((wl.batch, wl.B), dtype=torch.int32, device=dev)
    st = torch.empty((wl.batch, wl.B, 6), dtype=torch.float32, device=dev)
    ws = B.draft_workspace(head, wl.batch, wl.B, dev)
    path = head.path(wl.batch, wl.B, L.dtype, False)

    def call(_):
        B.draft_block(head, L, last, None, 1.0, wl.alphas[0], 0.0, out=(tok, st), workspace=ws, exclusive_device=True)

    for i in range(5):
        call(i)
    us = per_call_us(call, n, torch)
    assert path != 1 or B.workspace_error(ws) == 0, "persistent kernel reported an error"
    med = pct(us, 50)
    alg, _ = algorithmic_bytes(wl, 2 if wl.dtype == "bf16" else 4)
    comp = compulsory_bytes(wl, 2 if wl.dtype == "bf16" else 4)
    return {"batch": wl.batch, "B": wl.B, "V": V, "d": d, "H": H, "r": r, "dtype": wl.dtype,
            "path": "persistent" if path == 1 else "per-position launches", "us_per_block": dist(us),
            "tokens_per_s": round(wl.batch * wl.B / (med * 1e-6), 1), "us_per_position": round(med / wl.B, 2),
            "algorithmic_bytes_per_block": alg, "roofline_frac": round(alg / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "compulsory_frac": round(comp / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "tflops": round(method_flops(wl) / (med * 1e-6) / 1e12, 2)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="b64-d5120")
    ap.add_argument("--init", default="stress", choices=["baseline", "stress"])
    ap.add_argument("--alpha", type=float, default=0.5)
    ap.add_argument("--calls", type=int, default=100, help="calls per timing distribution (warm and cold)")
    ap.add_argument("--cold-mb", type=int, default=1024, help="scratch written between cold calls (MiB)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="single-thread oracle sample length")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="only the step, the roofline and the oracle leg")
    ap.add_argument("--profile-only", action="store_true",
                    help="for hardware-counter runs: only --steps draft blocks and a 1 GiB device copy "
                         "(the copy calibrates the HBM byte counters); no JSON line")
    ap.add_argument("--cooperative", action="store_true",
                    help="launch the persistent kernel cooperatively in the timed step (default: an ordinary "
                         "dispatch, DLS_EXCLUSIVE_DEVICE, since this process owns the device)")
    ap.add_argument("--no-cooperative-comparison", action="store_true",
                    help="leave out the timing of the other launch mode (a profiled run without cooperative launches)")
    ap.add_argument("--oracle-leg", help=argparse.SUPPRESS)
    ap.add_argument("--oracle-parity", action="store_true", help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.oracle_leg:
        oracle_leg(args)
        return
    EXC = not args.cooperative
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build measures one GPU only (the drafting path has no multi-GPU form "
              "here); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_07409_amd import binding as B
    from paper_2607_07409_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = W.WORKLOADS[args.workload]
    log(f"generating {wl.name} inputs ({args.init} weights)")
    hw = W.make_head(wl, args.init)
    long_h = W.make_long_logits(wl)
    last = W.make_last_token(wl)
    head = B.LocalHead.from_weights(hw, dev)
    log("preparing the head (folded input table, operand-ordered weights)")
    head.prepare()
    torch.cuda.synchronize()
    L = B.as_tensor(long_h, dev)
    path = head.path(wl.batch, wl.B, L.dtype, False)
    log(f"draft path: {'persistent' if path == 1 else 'per-position launches'}")
    last_t = torch.from_numpy(last).to(dev)
    tok = torch.empty((wl.batch, wl.B), dtype=torch.int32, device=dev)
    st = torch.empty((wl.batch, wl.B, 6), dtype=torch.float32, device=dev)
    ws = B.draft_workspace(head, wl.batch, wl.B, dev)

    def draft(_=None, exclusive=EXC):
        B.draft_block(head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st), workspace=ws,
                      exclusive_device=exclusive)

    if args.profile_only:
        for _ in range(args.steps):
            draft()
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)      # 1 GiB read + 1 GiB written per copy
        torch.cuda.synchronize()
        assert B.workspace_error(ws) == 0, "persistent kernel reported an error"
        log(f"profile run done: {args.steps} draft blocks of {wl.name}, 3 copies of 1 GiB")
        return

    # ---- one untimed draft: its tokens define the targets and feed the oracle's parity replay ----
    draft()
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0, "persistent kernel reported an error"
    g_tok = tok.cpu().numpy().copy()
    g_st = st.cpu().numpy().copy()
    targets, _ = W.make_targets(g_tok, wl)
    tgt = torch.from_numpy(targets).to(dev)
    acc = torch.empty(wl.batch, dtype=torch.int32, device=dev)
    B.accept_len(tok, tgt, out=acc)
    torch.cuda.synchronize()
    g_acc = acc.cpu().numpy().copy()

    # ---- the timed step (the driver's contract) ---------------------------------------------------
    def step():
        draft()
        B.accept_len(tok, tgt, out=acc)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = e0.elapsed_time(e1) / args.steps
    tokens_per_s = wl.batch * wl.B / (ms_step * 1e-3)
    assert B.workspace_error(ws) == 0, "persistent kernel reported an error"
    log(f"step {ms_step * 1e3:.1f} us ({wall:.2f} s wall) -> {tokens_per_s:.0f} drafted tokens/s")

    # ---- the dominant kernel: per-call distributions, warm and cold -------------------------------
    warm = per_call_us(draft, args.calls, torch)
    scratch = torch.empty(args.cold_mb << 20, dtype=torch.uint8, device=dev)
    cold = per_call_us(draft, args.calls, torch, scratch=scratch)
    del scratch
    assert B.workspace_error(ws) == 0, "persistent kernel reported an error"
    blk_us = sum(warm) / len(warm)
    alg_block, alg_step = algorithmic_bytes(wl)
    comp = compulsory_bytes(wl)
    flops = method_flops(wl)
    achieved = alg_block / (blk_us * 1e-6) / 1e9
    traffic = measured_traffic(wl.name) if path == 1 else None
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic["traffic_bytes_per_launch"] if traffic else None,
                "kernel": "k_draft_persistent (one launch per block)" if path == 1 else
                          "dls_draft_block (all launches of one block)",
                "us_per_launch": round(blk_us, 2),
                "algorithmic_bytes_per_launch": alg_block,
                "algorithmic_basis": "re-read formulation: per position W_vocab, W_ih, W_hh and W_rank plus one "
                                     "embedding row and one long-logit row per sequence; x B positions per launch",
                "compulsory_bytes_per_launch": comp,
                "compulsory_frac": round(comp / (blk_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                "measured_traffic_frac": (round(traffic["traffic_bytes_per_launch"] / (blk_us * 1e-6) / 1e9
                                                / HBM_PEAK_GBS, 4) if traffic else None),
                "us_per_position": round(blk_us / wl.B, 2),
                "matrix_tflops": round(flops / (blk_us * 1e-6) / 1e12, 2),
                "matrix_frac_of_bf16_peak": round(flops / (blk_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
                "timing": {"warm": dist(warm), "cold": dist(cold), "cold_scratch_mib": args.cold_mb}}
    log(f"draft block warm median {pct(warm, 50):.1f} us (p10 {pct(warm, 10):.1f}, p90 {pct(warm, 90):.1f}); "
        f"cold median {pct(cold, 50):.1f} us; {achieved:.0f} GB/s re-read algorithmic "
        f"({achieved / HBM_PEAK_GBS:.1%}), compulsory {roofline['compulsory_frac']:.1%}")

    peaks = measured_peaks(B, dev, torch)
    roofline["frac_of_measured_read_peak"] = round(achieved / peaks["hbm_read_GBs"], 4)
    log(f"measured peaks: HBM read {peaks['hbm_read_GBs']:.0f} GB/s (checksum ok={peaks['read_checksum_ok']}), "
        f"bf16 MFMA {peaks['bf16_mfma_TFLOPs']:.0f} TFLOP/s (exact={peaks['mfma_exact']}); the draft block "
        f"reaches {roofline['frac_of_measured_read_peak']:.1%} of the measured read rate")

    extras = {}
    if not args.no_extras:
        # the other launch mode (cooperative vs ordinary dispatch)
        if not args.no_cooperative_comparison:
            for _ in range(3):
                draft(exclusive=not EXC)
            other = per_call_us(lambda i: draft(exclusive=not EXC), 30, torch)
            extras["draft_block_" + ("cooperative" if EXC else "ordinary") + "_launch_us"] = dist(other)
            log(f"draft block with {'a cooperative' if EXC else 'an ordinary'} launch: {pct(other, 50):.1f} us")
        # the same block without row statistics (Algorithm 1 needs only the tokens): the kernel
        # then skips the statistics reduction and publish of every M tile
        tonly = per_call_us(lambda i: B.draft_block(head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, None),
                                                    workspace=ws, exclusive_device=EXC), 30, torch)
        extras["draft_block_tokens_only_us"] = dist(tonly)
        log(f"draft block without row statistics: {pct(tonly, 50):.1f} us")
        # the same block through the per-position launches (no prepared head)
        base_head = B.LocalHead(head.emb, head.w_ih, head.w_hh, head.w_rank, head.w_vocab)
        ws2 = B.draft_workspace(base_head, wl.batch, wl.B, dev)
        pp = per_call_us(lambda i: B.draft_block(base_head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st),
                                                 workspace=ws2), 10, torch)
        extras["draft_block_per_position_launches_us"] = dist(pp)
        log(f"per-position launches: {pct(pp, 50):.1f} us per block")
        del ws2, base_head
        # temperature sampling (T = 1, Gumbel-max with Philox noise) on the same block
        sm = per_call_us(lambda i: B.draft_block(head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st),
                                                 workspace=ws, exclusive_device=EXC, temperature=1.0,
                                                 seed=12345 + i), 30, torch)
        assert B.workspace_error(ws) == 0
        extras["sampling"] = {"temperature": 1.0, "us_per_block": dist(sm),
                              "tokens_per_s": round(wl.batch * wl.B / (pct(sm, 50) * 1e-6), 1),
                              "overhead_vs_greedy": round(pct(sm, 50) / pct(warm, 50) - 1.0, 4)}
        log(f"sampling at T = 1: {pct(sm, 50):.1f} us per block")
        # adaptive fusion (weights gated by the entropy of the long logits): the pre-pass over the
        # batch * B long-logit rows, then the gated draft; and the pre-pass alone (HBM-bound)
        unc = torch.empty((wl.batch, wl.B, 4), dtype=torch.float32, device=dev)
        rule = (B.UNC_ENTROPY, 0.4, 0.8)
        for _ in range(3):
            B.draft_block(head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st), workspace=ws,
                          exclusive_device=EXC, adaptive=rule, out_uncertainty=unc)
        ad = per_call_us(lambda i: B.draft_block(head, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st),
                                                 workspace=ws, exclusive_device=EXC, adaptive=rule,
                                                 out_uncertainty=unc), 30, torch)
        assert B.workspace_error(ws) == 0
        uws = torch.empty(max(256, B.long_uncertainty_workspace_size(wl.batch * wl.B, wl.V)), dtype=torch.uint8,
                          device=dev)
        un = per_call_us(lambda i: B.long_uncertainty(L, *rule, out=unc, workspace=uws), 50, torch)
        u_bytes = wl.batch * wl.B * (wl.V * L.element_size() + 16)
        u_gbs = u_bytes / (pct(un, 50) * 1e-6) / 1e9
        extras["adaptive_fusion"] = {
            "rule": "gate = clamp((H(p_L) / log V - 0.4) / 0.4, 0, 1) on alpha and beta",
            "us_per_block": dist(ad), "tokens_per_s": round(wl.batch * wl.B / (pct(ad, 50) * 1e-6), 1),
            "overhead_vs_greedy": round(pct(ad, 50) / pct(warm, 50) - 1.0, 4),
            "gate_mean": round(float(unc[..., 3].mean()), 4),
            "uncertainty_pass": {"rows": wl.batch * wl.B, "us_per_call": dist(un), "algorithmic_bytes": u_bytes,
                                 "achieved_GBs": round(u_gbs, 1), "frac_of_hbm_peak": round(u_gbs / HBM_PEAK_GBS, 4),
                                 "frac_of_measured_read_peak": round(u_gbs / peaks["hbm_read_GBs"], 4)}}
        log(f"adaptive fusion: {pct(ad, 50):.1f} us per block; uncertainty pass {pct(un, 50):.1f} us "
            f"({u_gbs / HBM_PEAK_GBS:.1%} of HBM peak)")
        del uws
        # the Markov local head (App. A) on the same workload: rho = E_M[previous token]
        import math
        em, wm = W.make_markov_head(wl.V, wl.r, "bf16", wl.seed, scale=math.sqrt(3.0 / math.sqrt(wl.r)))
        mhead = B.LocalHead.markov_from_weights(em, wm, dev).prepare()
        mws = B.draft_workspace(mhead, wl.batch, wl.B, dev)
        for _ in range(3):
            B.draft_block(mhead, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st), workspace=mws,
                          exclusive_device=EXC)
        mk = per_call_us(lambda i: B.draft_block(mhead, L, last_t, None, 1.0, args.alpha, 0.0, out=(tok, st),
                                                 workspace=mws, exclusive_device=EXC), 30, torch)
        assert B.workspace_error(mws) == 0
        extras["markov_head"] = {"head": "markov (E_M, W_M: V x r bf16)", "r": wl.r, "us_per_block": dist(mk),
                                 "tokens_per_s": round(wl.batch * wl.B / (pct(mk, 50) * 1e-6), 1)}
        log(f"markov head: {pct(mk, 50):.1f} us per block")
        del mhead, mws
        # unigram log-prior estimation (App. A) from a Zipf-distributed token stream
        n_p = 1 << 26
        ptok = torch.from_numpy(W.make_token_stream(n_p, wl.V, 5)).to(dev)
        plogp = torch.empty(wl.V, dtype=torch.float32, device=dev)
        pcnt = torch.empty(wl.V + 1, dtype=torch.int64, device=dev)
        for _ in range(3):
            B.unigram_log_prior(ptok, wl.V, 1.0, out=(plogp, pcnt))
        pr = per_call_us(lambda i: B.unigram_log_prior(ptok, wl.V, 1.0, out=(plogp, pcnt)), 10, torch)
        extras["prior_estimation"] = {"tokens": n_p, "V": wl.V, "us_per_call": dist(pr),
                                      "input_GBs": round(4 * n_p / (pct(pr, 50) * 1e-6) / 1e9, 1)}
        log(f"unigram prior over {n_p} tokens: {pct(pr, 50):.1f} us")
        del ptok
        # standalone fused combine at the two serving shapes, cold (rotating >= 1 GB of inputs)
        combine = {}
        for R in (256, 1024):
            Lc = B.as_tensor(W.make_logit_rows(R, wl.V, "bf16", 77, "onehot", 3.0, purpose=20), dev)
            Sc = B.as_tensor(W.make_logit_rows(R, wl.V, "bf16", 77, "normal", 2.0, purpose=21), dev)
            nbuf = max(2, int(np.ceil(1.0e9 / (Lc.numel() * 4))))
            bufs = [(Lc, Sc)] + [(Lc.clone(), Sc.clone()) for _ in range(nbuf - 1)]
            ctok = torch.empty(R, dtype=torch.int32, device=dev)
            cst = torch.empty((R, 6), dtype=torch.float32, device=dev)
            cws = torch.empty(max(256, B.combine_logits_workspace_size(R, wl.V)), dtype=torch.uint8, device=dev)
            c_bytes = R * wl.V * 2 * 2
            row = {"algorithmic_bytes": c_bytes, "buffers_rotated": nbuf}
            for name, so in (("tokens", None), ("tokens_and_stats", cst)):
                for i in range(5):
                    B.combine_logits(*bufs[i % nbuf], None, 1.0, args.alpha, 0.0, out=(ctok, so, None), workspace=cws)
                us = per_call_us(lambda i: B.combine_logits(*bufs[i % nbuf], None, 1.0, args.alpha, 0.0,
                                                            out=(ctok, so, None), workspace=cws), 60, torch)
                gbs = c_bytes / (pct(us, 50) * 1e-6) / 1e9
                row[name] = {"us_per_call": dist(us), "achieved_GBs": round(gbs, 1),
                             "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                             "frac_of_measured_read_peak": round(gbs / peaks["hbm_read_GBs"], 4)}
            combine[f"[{R}, {wl.V}]"] = row
            log(f"combine [{R}, {wl.V}]: tokens {row['tokens']['us_per_call']['median']:.1f} us "
                f"({row['tokens']['frac_of_hbm_peak']:.1%}; {row['tokens']['frac_of_measured_read_peak']:.1%} of "
                f"the measured read rate), with statistics "
                f"{row['tokens_and_stats']['us_per_call']['median']:.1f} us "
                f"({row['tokens_and_stats']['frac_of_hbm_peak']:.1%})")
            del bufs, Lc, Sc
        extras["combine"] = combine
        # every drafting workload, and the block-7 setting (a head trained at 16 serving B = 7)
        wls = {}
        del head, ws
        torch.cuda.empty_cache()
        cases = [(n, W.WORKLOADS[n]) for n in W.WORKLOAD_ORDER]
        cases.append(("qwen3-8b-b1-block7", W.WORKLOADS["qwen3-8b-b1"].with_(B=7)))
        # the ABI's largest batch: four persistent launches of 64 sequences on one workspace
        cases.append(("b256-d5120", W.WORKLOADS["b64-d5120"].with_(batch=256)))
        for name, w_ in cases:
            wls[name] = time_workload(B, W, w_, dev, torch)
            torch.cuda.empty_cache()
            r_ = wls[name]
            log(f"{name}: {r_['us_per_block']['median']:.1f} us per block ({r_['path']}) -> "
                f"{r_['tokens_per_s']:.0f} drafted tokens/s, {r_['roofline_frac']:.1%} of its re-read roofline, "
                f"{r_['tflops']} TFLOP/s")
        extras["workloads"] = wls

    # ---- CPU oracle leg (fresh subprocesses) and the element-by-element parity of the timed draft --
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        visited = np.unique(np.concatenate([last, g_tok.reshape(-1)]))
        fd, npz = tempfile.mkstemp(suffix=".npz", dir="/dev/shm" if os.path.isdir("/dev/shm") else None)
        os.close(fd)
        try:
            np.savez(npz, emb_tokens=visited, emb_rows=hw.emb.bits[visited] if hasattr(hw.emb, "bits") else
                     np.asarray(hw.emb)[visited], w_ih=getattr(hw.w_ih, "bits", hw.w_ih),
                     w_hh=getattr(hw.w_hh, "bits", hw.w_hh), w_rank=getattr(hw.w_rank, "bits", hw.w_rank),
                     w_vocab=getattr(hw.w_vocab, "bits", hw.w_vocab), long=getattr(long_h, "bits", long_h),
                     last=last, tokens=g_tok, stats=g_st, targets=targets, accept=g_acc, alpha=args.alpha)
            ncpu = len(os.sched_getaffinity(0))
            log(f"CPU oracle: every sequence with {ncpu} threads (parity), then a {args.cpu_seconds:.0f} s "
                f"single-thread sample")
            full = run_oracle_subprocess(npz, args, ncpu, parity=True)
            one = run_oracle_subprocess(npz, args, 1, parity=False)
        finally:
            os.unlink(npz)
        parity = full.pop("parity")
        cpu = {"value": round(full["tokens_per_s"], 3), "unit": "tokens/s", "cores": int(full["threads"]),
               "kind": "oracle",
               "sample": f"all {full['sequences']} sequences of one {wl.name} block (B={wl.B}) replayed on the GPU "
                         f"draft, float64 numpy, {full['seconds']:.1f} s wall, fresh process",
               "cpu_model": cpu_model(),
               "single_thread": {"value": round(one["tokens_per_s"], 3), "cores": int(one["threads"]),
                                 "sample": f"{one['sequences']} sequences, {one['seconds']:.1f} s wall"}}
        log(f"CPU oracle: {cpu['value']} tokens/s on {cpu['cores']} threads, "
            f"{cpu['single_thread']['value']} on 1; parity ok={parity['ok']} near_ties={parity['near_ties']}")

    out = {
        "metric": "drafted tokens/sec per block step; fused-combine HBM GB/s as % of peak",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "B": wl.B, "V": wl.V, "d": wl.d, "H": wl.H,
                   "r": wl.r, "weights": f"bf16 ({args.init} init)", "alpha": args.alpha, "beta": 0.0,
                   "step": "draft_block + accept_len",
                   "launch": "ordinary dispatch (DLS_EXCLUSIVE_DEVICE)" if EXC else "cooperative"},
        "roofline": roofline,
        "measured_peaks": peaks,
        "cpu_baseline": cpu,
        "parity": parity,
    }
    out.update(extras)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
