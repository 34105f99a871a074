"""Benchmark of the batched backoff query and the fused greedy step on one MI355X.

Workload (the 20M n-gram 6-gram model, V = 1024, synthetic and seeded): a
step is one ``advance`` launch over 128 independent batches of 512 hypotheses
(65,536 uniformly drawn states), writing scores [65536, 1024] fp32 and next
states [65536, 1024] int32 -- 512 MiB, more than the 256 MB Infinity Cache, so
the output really streams to HBM.  The value is (state, token) scores per
second over the timed steps.  The same run also reports:

* roofline: algorithmic HBM bytes per launch (library ``query_bytes``: output
  rows plus the records and arcs of chain states of order >= 2) divided by the
  mean kernel duration from HIP events on the launch stream, against 8 TB/s;
  ``traffic`` is the measured HBM bytes per launch from the committed rocprofv3
  counter summary when it was taken on the current kernel source, else null;
* latency of a single 512-hypothesis call (median of 100, the calls enqueued
  ahead of the GPU so that the events bracket device time; also the same
  with the GPU waiting for each call's submission, and the per-call time of
  100 calls back to back), with its algorithmic bytes as a fraction of the
  HBM roofline (roofline_b512_single);
* the same work as 128 separate 512-hypothesis calls on 8 streams, captured in
  one HIP graph, likewise against the roofline (roofline_b512_graph), with
  the host time of each replay call and the GPU's own time per replay when
  the replays are enqueued ahead of it;
* the transducer mode, one launch per step, at 32 and 256 hypotheses;
* the fused greedy CTC step at B = 256 utterances, 1025 classes, per frame,
  and the same decode of 1000 frames as one launch;
* the same decode at B = 4096 utterances x 200 frames, writing the labels,
  with its algorithmic HBM bytes (ASR rows, and chain records and arcs on the
  frames that consult the LM, counted from an untimed decode that also
  writes each frame's state), and the time of a decode that writes both;
* the k best fused tokens (beam expansion) of 1024 hypotheses, k = 4, 32 and 128;
* plain fusion on the 200k-n-gram 4-gram at B = 32 hypotheses x 200 steps;
* cpu_baseline: the CPU oracle on a bounded sample of the same workload, on all
  host cores; cpu_baseline_decode: the oracle on the whole CTC decode above,
  with whether its labels equal the GPU decode's.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "LM (state,token) scores/s + achieved HBM GB/s for batched advance; fused step/s"
PEAK_HBM_GBPS = 8000.0
KERNEL_SOURCES = ["paper_2505_22857_amd/csrc/advance.hip", "paper_2505_22857_amd/csrc/walk.h",
                  "paper_2505_22857_amd/csrc/trie.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "advance_6gram20m_traffic.md")


def kernel_source_hash() -> str:
    """Hash of the advance kernel's sources with comments and blank lines
    removed, so that the committed counters stay valid across comment edits."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            src = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        lines = [re.sub(r"//.*", "", ln).rstrip() for ln in src.splitlines()]
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


def committed_traffic():
    """Measured HBM bytes per launch from the counter summary, if it matches this kernel."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    txt = open(TRAFFIC_FILE).read()
    m_hash = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", txt)
    m_val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not m_hash or not m_val or m_hash.group(1) != kernel_source_hash():
        return None
    return float(m_val.group(1))


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batches", type=int, default=128, help="512-hypothesis batches per step")
    ap.add_argument("--fused-frames", type=int, default=1000)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target oracle time; 0 skips")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 512 MiB device copy and fill (counter calibration)")
    ap.add_argument("--advance-only", action="store_true", help="skip the fused step and the oracle")
    ap.add_argument("--no-graph", action="store_true", help="skip the graph of 512-hypothesis calls")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (a multi-GPU run would "
              "replicate the trie and split the batch, with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2505_22857_amd as ng
    from synth import WORKLOADS, make_model, seed_for, uniform_states

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    spec = WORKLOADS["sixgram_20m"]
    t0 = time.time()
    model = make_model("sixgram_20m")
    log(f"model generated in {time.time() - t0:.1f}s: counts {model.counts}")
    t0 = time.time()
    lm = ng.NgpuLM.from_model(model)
    log(f"trie built in {time.time() - t0:.1f}s: {lm.num_states} states, {lm.num_arcs} arcs, "
        f"{lm.device_bytes / 2**20:.1f} MiB")
    lm.upload(dev)
    V = lm.vocab_size
    Bb = spec.batch
    R = args.batches
    B = R * Bb
    states_np = uniform_states(model, B, seed=seed_for("sixgram_20m") + 1000)
    states = torch.from_numpy(states_np).to(dev)
    scores = torch.empty((B, V), dtype=torch.float32, device=dev)
    nxt = torch.empty((B, V), dtype=torch.int32, device=dev)
    hbm_bytes, total_bytes = lm.query_bytes(states_np)
    stream = torch.cuda.current_stream()

    if args.copy_calibration:
        # reference kernels of known traffic: a 512 MiB device copy and a 512 MiB fill
        src = torch.empty(2**29 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        dst.copy_(src)
        c0.record(stream)
        for _ in range(5):
            dst.copy_(src)
        c1.record(stream)
        torch.cuda.synchronize()
        cp_ms = c0.elapsed_time(c1) / 5
        c0.record(stream)
        for _ in range(5):
            dst.fill_(2.0)
        c1.record(stream)
        torch.cuda.synchronize()
        fill_ms = c0.elapsed_time(c1) / 5
        log(f"reference: 512 MiB copy {cp_ms:.3f} ms ({2 * 2**29 / cp_ms / 1e6:.0f} GB/s read+write), "
            f"512 MiB fill {fill_ms:.3f} ms ({2**29 / fill_ms / 1e6:.0f} GB/s)")
        del src, dst

    # ---- single 512-hypothesis call latency
    s512, n512 = scores[:Bb], nxt[:Bb]
    for _ in range(10):
        lm.advance(states[:Bb], s512, n512)
    torch.cuda.synchronize()

    def single_calls(queued):
        # queued: the GPU first spins for a few ms, so the host enqueues all
        # calls ahead and each event pair brackets the call's device time only;
        # otherwise the GPU waits for each call's host-side submission, which
        # the bracket then includes
        views = [(states[sl], scores[sl], nxt[sl]) for sl in
                 (slice((r % R) * Bb, (r % R + 1) * Bb) for r in range(100))]
        lat = []
        if queued:
            torch.cuda._sleep(int(8e6))
        for st_r, sc_r, nx_r in views:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            lm.advance(st_r, sc_r, nx_r)
            e1.record(stream)
            lat.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) * 1e3 for a, b in lat]))

    lat_host_us = single_calls(False)
    lat_us = single_calls(True)
    # the same 100 calls enqueued back to back with no events between them,
    # timed as a whole: the per-call cost of a stream of dependent-free calls
    views = [(states[sl], scores[sl], nxt[sl]) for sl in
             (slice((r % R) * Bb, (r % R + 1) * Bb) for r in range(100))]
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(int(8e6))
    b0.record(stream)
    for st_r, sc_r, nx_r in views:
        lm.advance(st_r, sc_r, nx_r)
    b1.record(stream)
    torch.cuda.synchronize()
    b2b_us = b0.elapsed_time(b1) * 1e3 / len(views)
    log(f"single B={Bb} call: median {lat_us:.1f} us of device time ({lat_host_us:.1f} us paced by the host); "
        f"{b2b_us:.1f} us per call back to back")
    # algorithmic bytes of one 512-hypothesis call: the mean over the slices the 100 calls cycle through
    call_bytes = float(np.mean([lm.query_bytes(states_np[(r % R) * Bb:(r % R + 1) * Bb])[0] for r in range(100)]))
    single = {"bound": "hbm", "achieved": call_bytes / (lat_us * 1e-6) / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
              "frac": call_bytes / (lat_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, "bytes_per_call": call_bytes,
              "us_per_call": lat_us, "us_per_call_host_paced": lat_host_us, "us_per_call_back_to_back": b2b_us,
              "workload": f"one advance call of B={Bb} uniform states (median of 100, HIP events around each "
                          f"call, enqueued ahead of the GPU; us_per_call_host_paced: the GPU idle until each "
                          f"call is submitted; us_per_call_back_to_back: 100 calls enqueued ahead with no "
                          f"events between them, timed as a whole)"}

    # ---- sustained: one launch over all R batches per step
    for _ in range(args.warmup):
        lm.advance(states, scores, nxt)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        lm.advance(states, scores, nxt)
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    assert lm.check_states() == 0
    kern_ms = np.array([a.elapsed_time(b) for a, b in ev])
    mean_ms = float(kern_ms.mean())
    ms_per_step = wall * 1e3 / args.steps
    value = B * V * args.steps / wall
    achieved = hbm_bytes / (mean_ms * 1e-3) / 1e9
    log(f"advance B={B}: wall {ms_per_step:.3f} ms/step, kernel mean {mean_ms:.3f} ms "
        f"(min {kern_ms.min():.3f}), {achieved:.0f} GB/s algorithmic HBM, "
        f"{total_bytes / (mean_ms * 1e-3) / 1e9:.0f} GB/s incl. cache-resident rows")

    # ---- the same work as R separate 512-hypothesis calls in one HIP graph over 8 streams
    graph = None
    if not args.no_graph:
        streams = [torch.cuda.Stream() for _ in range(8)]

        def fan_out():
            main_s = torch.cuda.current_stream()
            for i, st_ in enumerate(streams):
                st_.wait_stream(main_s)
                with torch.cuda.stream(st_):
                    for r in range(i, R, len(streams)):
                        sl = slice(r * Bb, (r + 1) * Bb)
                        lm.advance(states[sl], scores[sl], nxt[sl])
            for st_ in streams:
                main_s.wait_stream(st_)

        fan_out()                                   # eager once on the same streams
        torch.cuda.synchronize()
        g_adv = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_adv):
            fan_out()
        for _ in range(3):
            g_adv.replay()
        torch.cuda.synchronize()
        reps = 20
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t_host = time.perf_counter()
        g0.record(stream)
        for _ in range(reps):
            g_adv.replay()
        g1.record(stream)
        host_ms = (time.perf_counter() - t_host) * 1e3 / reps
        torch.cuda.synchronize()
        g_ms = g0.elapsed_time(g1) / reps
        # the same replays enqueued while the GPU spins, so they run back to
        # back at the GPU's own pace: valid only if the host finished
        # enqueueing before the spin ended
        gs = torch.cuda.Event(enable_timing=True)
        gs.record(stream)
        torch.cuda._sleep(int(4e7))
        g0.record(stream)
        t_host = time.perf_counter()
        for _ in range(reps):
            g_adv.replay()
        enqueue_ms = (time.perf_counter() - t_host) * 1e3
        g1.record(stream)
        torch.cuda.synchronize()
        spin_ms = gs.elapsed_time(g0)
        q_ms = g0.elapsed_time(g1) / reps
        assert lm.check_states() == 0
        graph = {"workload": f"{R} calls of B={Bb} on 8 streams, one HIP graph replay",
                 "bound": "hbm", "achieved": hbm_bytes / (g_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                 "frac": hbm_bytes / (g_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, "bytes_per_replay": hbm_bytes,
                 "ms": g_ms, "scores_per_s": B * V / (g_ms * 1e-3),
                 "host_ms_per_replay_call": host_ms,
                 "ms_queued": q_ms if enqueue_ms < spin_ms else None,
                 "frac_queued": (hbm_bytes / (q_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS) if enqueue_ms < spin_ms else None,
                 "method": "20 replays back to back between HIP events (ms, frac); host_ms_per_replay_call: "
                           "host time of one replay call in that loop; ms_queued / frac_queued: the 20 "
                           "replays enqueued while the GPU spins, then timed on the GPU alone"}
        log(f"advance as {R} graph-captured B={Bb} calls on 8 streams: {g_ms:.3f} ms per replay "
            f"(host {host_ms:.3f} ms per replay call), {graph['scores_per_s']:.3g} scores/s; "
            f"queued ahead: {q_ms:.3f} ms per replay (enqueue {enqueue_ms:.1f} ms, spin {spin_ms:.1f} ms)")
        del g_adv

    if args.advance_only:
        return

    # ---- fused greedy CTC step (256 utterances x 1000 frames on the 20M 6-gram), per frame
    fspec = WORKLOADS["ctc_b256_t1000"]
    Bf, T = fspec.batch, args.fused_frames
    g = torch.Generator(device=dev)
    g.manual_seed(seed_for("ctc_b256_t1000"))
    logits = torch.randn((T, Bf, V + 1), generator=g, device=dev, dtype=torch.float32) * 3.0
    logits[..., V] += fspec.blank_boost
    asr = torch.log_softmax(logits, dim=-1)
    del logits
    fst = torch.zeros(Bf, dtype=torch.int32, device=dev)
    prev = torch.full((Bf,), V, dtype=torch.int32, device=dev)
    tok = torch.empty(Bf, dtype=torch.int32, device=dev)
    for t in range(min(T, 20)):
        lm.fused_greedy_step(asr[t], fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, tokens=tok)
    fst.zero_()
    prev.fill_(V)
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rows = list(asr.unbind(0))   # the per-frame row views, made before the timed loop
    f0.record(stream)
    for t in range(T):
        lm.fused_greedy_step(rows[t], fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, tokens=tok)
    f1.record(stream)
    torch.cuda.synchronize()
    f_ms = f0.elapsed_time(f1)
    assert lm.check_states() == 0
    fused = {"workload": f"CTC, B={Bf} utterances x {T} frames, {V + 1} classes, lambda={fspec.lam}, "
                         "one launch per frame",
             "steps_per_s": T / (f_ms * 1e-3), "frames_per_s": Bf * T / (f_ms * 1e-3),
             "us_per_step": f_ms * 1e3 / T}
    log(f"fused CTC: {fused['us_per_step']:.1f} us/step, {fused['frames_per_s']:.3g} frames/s")

    # ---- transducer mode, one launch per step (the LM consulted on non-blank frames), B = 32 and 256
    Tt = min(T, 200)
    transducer = {"workload": f"transducer, 20M 6-gram, {V + 1} classes (log_softmax of N(0,3) logits, blank +"
                              f"{fspec.blank_boost}), lambda={fspec.lam}, one launch per step, {Tt} steps"}
    for Bt in (32, 256):
        tst = torch.zeros(Bt, dtype=torch.int32, device=dev)
        ttok = torch.empty((Tt, Bt), dtype=torch.int32, device=dev)
        trows = [asr[t, :Bt] for t in range(Tt)]
        for t in range(min(20, Tt)):
            lm.fused_greedy_step(trows[t], fspec.lam, tst, mode=ng.NGPU_FUSION_TRANSDUCER, tokens=ttok[t])
        tst.zero_()
        torch.cuda.synchronize()
        f0.record(stream)
        for t in range(Tt):
            lm.fused_greedy_step(trows[t], fspec.lam, tst, mode=ng.NGPU_FUSION_TRANSDUCER, tokens=ttok[t])
        f1.record(stream)
        torch.cuda.synchronize()
        transducer[f"b{Bt}_us_per_step"] = f0.elapsed_time(f1) * 1e3 / Tt
        transducer[f"b{Bt}_lm_share"] = float((ttok != V).float().mean())
    assert lm.check_states() == 0
    log(f"fused transducer: {transducer['b32_us_per_step']:.1f} us/step at B=32, "
        f"{transducer['b256_us_per_step']:.1f} us/step at B=256")

    # ---- the same per-frame launches replayed from one HIP graph (decoding steps in a graph)
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):             # warm the launch path on the capture stream
            for t in range(3):
                lm.fused_greedy_step(asr[t], fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, tokens=tok)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g_steps = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_steps):
            for t in range(T):
                lm.fused_greedy_step(asr[t], fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, tokens=tok)
        g_ms = []
        for _ in range(3):
            fst.zero_()
            prev.fill_(V)
            f0.record(stream)
            g_steps.replay()
            f1.record(stream)
            torch.cuda.synchronize()
            g_ms.append(f0.elapsed_time(f1))
        assert lm.check_states() == 0
        fused["graph_us_per_step"] = float(np.median(g_ms)) * 1e3 / T
        log(f"fused CTC, {T} per-frame launches in one graph: {fused['graph_us_per_step']:.2f} us/step")
        del g_steps

    # ---- the same decode as one launch over all frames
    asr_bt = asr.permute(1, 0, 2)            # [B, T, C] view, unit class stride
    labels = torch.empty((Bf, T), dtype=torch.int32, device=dev)
    fst.zero_()
    prev.fill_(V)
    lm.fused_greedy_decode(asr_bt, fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, labels=labels)
    torch.cuda.synchronize()
    d_ms = []
    for _ in range(3):
        fst.zero_()
        prev.fill_(V)
        f0.record(stream)
        lm.fused_greedy_decode(asr_bt, fspec.lam, fst, prev, mode=ng.NGPU_FUSION_CTC, labels=labels)
        f1.record(stream)
        torch.cuda.synchronize()
        d_ms.append(f0.elapsed_time(f1))
    assert lm.check_states() == 0
    dm = float(np.median(d_ms))
    fused_decode = {"workload": f"CTC, B={Bf} utterances x {T} frames, {V + 1} classes, lambda={fspec.lam}, "
                                "one launch for all frames",
                    "ms": dm, "steps_per_s": T / (dm * 1e-3), "frames_per_s": Bf * T / (dm * 1e-3),
                    "us_per_step": dm * 1e3 / T}
    log(f"fused CTC decode in one launch: {dm:.2f} ms, {fused_decode['us_per_step']:.2f} us/step, "
        f"{fused_decode['frames_per_s']:.3g} frames/s")
    # ---- a large batch: 4096 utterances x 200 frames, where the decode is bandwidth-bound
    Bl, Tl = 4096, 200
    gl_ = torch.Generator(device=dev)
    gl_.manual_seed(seed_for("ctc_b256_t1000") + 20)
    lasr = torch.log_softmax(torch.randn((Bl, Tl, V + 1), generator=gl_, device=dev) * 3.0
                             + torch.nn.functional.one_hot(torch.tensor(V, device=dev), V + 1) * fspec.blank_boost,
                             dim=-1)
    lst_ = torch.zeros(Bl, dtype=torch.int32, device=dev)
    lprev = torch.full((Bl,), V, dtype=torch.int32, device=dev)
    llab = torch.empty((Bl, Tl), dtype=torch.int32, device=dev)
    lls = torch.empty((Bl, Tl), dtype=torch.int32, device=dev)
    # one untimed decode that also writes each frame's state (for the byte count below); the timed
    # decodes write the labels only, as a decoder would
    lm.fused_greedy_decode(lasr, fspec.lam, lst_, lprev, mode=ng.NGPU_FUSION_CTC, labels=llab, label_states=lls)
    llab2 = torch.empty_like(llab)
    for _ in range(4):   # warm-up: the first launches of this decode run slower
        lst_.zero_()
        lprev.fill_(V)
        lm.fused_greedy_decode(lasr, fspec.lam, lst_, lprev, mode=ng.NGPU_FUSION_CTC, labels=llab2)
    torch.cuda.synchronize()
    l_ms = []
    for _ in range(10):
        lst_.zero_()
        lprev.fill_(V)
        f0.record(stream)
        lm.fused_greedy_decode(lasr, fspec.lam, lst_, lprev, mode=ng.NGPU_FUSION_CTC, labels=llab2)
        f1.record(stream)
        torch.cuda.synchronize()
        l_ms.append(f0.elapsed_time(f1))
    lst_.zero_()
    lprev.fill_(V)
    f0.record(stream)
    lm.fused_greedy_decode(lasr, fspec.lam, lst_, lprev, mode=ng.NGPU_FUSION_CTC, labels=llab2, label_states=lls)
    f1.record(stream)
    torch.cuda.synchronize()
    ls_ms = f0.elapsed_time(f1)
    assert lm.check_states() == 0
    assert torch.equal(llab, llab2)
    lm_ms = float(np.median(l_ms))
    # algorithmic HBM bytes: every frame's ASR row, plus on frames that consult the LM (not blank,
    # not the repeat) the chain record and arcs of the state the frame starts in
    lab_h, st_h = llab.cpu().numpy(), lls.cpu().numpy()
    prev_lab = np.concatenate([np.full((Bl, 1), V, np.int32), lab_h[:, :-1]], axis=1)
    start_st = np.concatenate([np.zeros((Bl, 1), np.int32), st_h[:, :-1]], axis=1)
    lm_frames = (lab_h != V) & (lab_h != prev_lab)
    lm_states = start_st[lm_frames]
    chain_bytes = lm.query_bytes(lm_states)[0] - 8 * V * len(lm_states)
    dec_bytes = Bl * Tl * 4 * (V + 1) + chain_bytes
    fused_large = {"workload": f"CTC, B={Bl} utterances x {Tl} frames, {V + 1} classes, lambda={fspec.lam}, "
                               "one launch writing the labels (median of 10)",
                   "ms": lm_ms, "ms_with_label_states": ls_ms, "frames_per_s": Bl * Tl / (lm_ms * 1e-3),
                   "lm_frame_share": float(lm_frames.mean()),
                   "algorithmic_bytes": int(dec_bytes), "algorithmic_gbps": dec_bytes / (lm_ms * 1e-3) / 1e9}
    log(f"fused CTC decode, B={Bl} x {Tl}: {lm_ms:.2f} ms, {fused_large['frames_per_s']:.3g} frames/s, "
        f"{fused_large['algorithmic_gbps']:.0f} GB/s algorithmic (LM on {100 * lm_frames.mean():.0f} % of frames); "
        f"{ls_ms:.2f} ms also writing each frame's state; the 10 runs {np.round(l_ms, 3).tolist()}")
    del lasr, llab, llab2, lls

    asr_host = asr_bt.contiguous().cpu().numpy() if args.cpu_seconds > 0 else None   # for the oracle's decode
    gpu_labels = labels.cpu().numpy()
    del asr, asr_bt

    # ---- beam expansion on the 20M 6-gram: the k best fused tokens of 1024 hypotheses
    Bk = 1024
    kst = torch.from_numpy(uniform_states(model, Bk, seed=seed_for("ctc_b256_t1000") + 9)).to(dev)
    gk = torch.Generator(device=dev)
    gk.manual_seed(seed_for("ctc_b256_t1000") + 10)
    kasr = torch.log_softmax(torch.randn((Bk, V), generator=gk, device=dev) * 3.0, dim=-1)
    topk = {"workload": f"{Bk} hypotheses (256 utterances x beam 4), V={V}, 20M 6-gram, lambda={fspec.lam}"}
    for kk in (4, 32, 128):
        ktok = torch.empty((Bk, kk), dtype=torch.int32, device=dev)
        ksc = torch.empty((Bk, kk), dtype=torch.float32, device=dev)
        knx = torch.empty((Bk, kk), dtype=torch.int32, device=dev)
        for _ in range(5):
            lm.fused_topk(kasr, fspec.lam, kk, kst, tokens=ktok, scores=ksc, next_states=knx)
        torch.cuda.synchronize()
        f0.record(stream)
        for _ in range(50):
            lm.fused_topk(kasr, fspec.lam, kk, kst, tokens=ktok, scores=ksc, next_states=knx)
        f1.record(stream)
        torch.cuda.synchronize()
        topk[f"k{kk}_us_per_call"] = f0.elapsed_time(f1) * 1e3 / 50
    assert lm.check_states() == 0
    log(f"fused top-k over {Bk} hypotheses: k=4 {topk['k4_us_per_call']:.1f} us, "
        f"k=32 {topk['k32_us_per_call']:.1f} us, k=128 {topk['k128_us_per_call']:.1f} us per call")
    del kasr

    # ---- plain fusion on the 200k 4-gram: B = 32 hypotheses x 200 steps
    pspec = WORKLOADS["fourgram_200k"]
    pmodel = make_model("fourgram_200k")
    plm = ng.NgpuLM.from_model(pmodel).upload(dev)
    Bp, Tp = pspec.batch, pspec.steps
    gp = torch.Generator(device=dev)
    gp.manual_seed(seed_for("fourgram_200k"))
    pasr = torch.log_softmax(torch.randn((Tp, Bp, V), generator=gp, device=dev) * 3.0, dim=-1)
    pstart = torch.from_numpy(uniform_states(pmodel, Bp, seed=seed_for("fourgram_200k") + 77)).to(dev)
    pst = pstart.clone()
    ptok = torch.empty(Bp, dtype=torch.int32, device=dev)
    for t in range(20):
        plm.fused_greedy_step(pasr[t], pspec.lam, pst, tokens=ptok)
    pst.copy_(pstart)
    torch.cuda.synchronize()
    prows = list(pasr.unbind(0))
    f0.record(stream)
    for t in range(Tp):
        plm.fused_greedy_step(prows[t], pspec.lam, pst, tokens=ptok)
    f1.record(stream)
    torch.cuda.synchronize()
    p_ms = f0.elapsed_time(f1)
    plabels = torch.empty((Bp, Tp), dtype=torch.int32, device=dev)
    pasr_bt = pasr.permute(1, 0, 2)
    pd = []
    for _ in range(4):
        pst.copy_(pstart)
        f0.record(stream)
        plm.fused_greedy_decode(pasr_bt, pspec.lam, pst, labels=plabels)
        f1.record(stream)
        torch.cuda.synchronize()
        pd.append(f0.elapsed_time(f1))
    assert plm.check_states() == 0
    pdm = float(np.median(pd[1:]))
    fused_plain = {"workload": f"plain fusion, 4-gram V={V} 200k n-grams, B={Bp} hypotheses x {Tp} steps, "
                               f"lambda={pspec.lam}",
                   "per_step_launch_us": p_ms * 1e3 / Tp, "one_launch_us_per_step": pdm * 1e3 / Tp,
                   "steps_per_s_one_launch": Tp / (pdm * 1e-3)}
    log(f"fused plain (B={Bp}): {fused_plain['per_step_launch_us']:.1f} us/step one launch per step, "
        f"{fused_plain['one_launch_us_per_step']:.2f} us/step in one decode launch")
    del plm, pasr, pasr_bt

    # ---- CPU oracle on a bounded sample of the same workload
    cpu = cpu_decode = None
    if args.cpu_seconds > 0:
        from oracle import Oracle
        cores = len(os.sched_getaffinity(0))
        o = Oracle.from_model(model)
        probe = states_np[:4096]
        t0 = time.perf_counter()
        o.advance(probe, nthreads=cores)
        dt = time.perf_counter() - t0
        n = int(min(1 << 22, max(4096, args.cpu_seconds / max(dt, 1e-6) * len(probe))))
        sample = uniform_states(model, n, seed=seed_for("sixgram_20m") + 1000)   # starts with the benchmark states
        t0 = time.perf_counter()
        o.advance(sample, nthreads=cores)
        dt = time.perf_counter() - t0
        cpu = {"value": n * V / dt, "unit": "scores/s", "cores": cores, "kind": "oracle",
               "sample": f"{n} uniform states of the same model (the benchmark draw extended), "
                         f"full {V}-token rows, {dt:.1f}s"}
        log(f"oracle: {cpu['value']:.3g} scores/s on {cores} cores")
        # the whole 256-utterance CTC decode (same ASR tensor as the GPU decode above)
        from oracle import MODE_CTC
        t0 = time.perf_counter()
        ol, _ = o.decode(asr_host, MODE_CTC, fspec.lam, np.zeros(Bf, np.int32), nthreads=cores)
        dt = time.perf_counter() - t0
        cpu_decode = {"value": Bf * T / dt, "unit": "utterance-frames/s", "cores": cores, "kind": "oracle",
                      "sample": f"the whole CTC decode of {Bf} utterances x {T} frames, {dt:.1f}s",
                      "labels_match_gpu": bool(np.array_equal(ol, gpu_labels))}
        log(f"oracle CTC decode: {cpu_decode['value']:.3g} frames/s on {cores} cores, "
            f"labels match the GPU decode: {cpu_decode['labels_match_gpu']}")
        del o, asr_host

    out = {
        "metric": METRIC, "value": value, "unit": "scores/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"6-gram V={V} 20M n-grams (trie {lm.device_bytes / 2**20:.0f} MiB), "
                               f"advance over {R} batches of {Bb} uniform states per launch",
                   "vocab": V, "order": model.max_order, "ngrams": model.num_ngrams,
                   "states": lm.num_states, "batch": Bb, "batches_per_step": R, "hyps_per_step": B},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS, "traffic": committed_traffic(),
                     "bytes_per_launch": hbm_bytes, "kernel_ms": mean_ms,
                     "total_bytes_per_launch": total_bytes,
                     "total_gbps": total_bytes / (mean_ms * 1e-3) / 1e9},
        "latency_b512_us": lat_us,
        "roofline_b512_single": single,
        "roofline_b512_graph": graph,
        "fused_transducer": transducer,
        "fused": fused,
        "fused_decode": fused_decode,
        "fused_decode_large": fused_large,
        "fused_plain": fused_plain,
        "fused_topk": topk,
        "cpu_baseline": cpu,
        "cpu_baseline_decode": cpu_decode,
        "kernel_source_sha256": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
