"""Throughput of the rotated W2A4 quantized linear on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-prefill] [--no-cpu]

Decode (the headline ``value``): LLaMA-3.1-8B-shaped layers (q 4096x4096, k and v 1024x4096, o
4096x4096, gate and up 14336x4096, down 4096x14336 with 7 Hadamard blocks of 2048), MNZ 2-bit
weights, M = 1 token, 32 distinct seeded layers per step (1.74 GB of packed words, so the weights
stream from HBM rather than the 256 MB Infinity Cache).  Per layer four linears with real data
dependencies: q|k|v and gate|up stacked along N since they share their input; o reads the q part of
the q|k|v output, gate|up reads the o output, down reads the gate part of the gate|up output, and the
next layer's q|k|v reads the down output (stand-ins for attention and the gated activation, which are
not part of the quantized linear).  Every linear rotates and quantizes its fp16 input.  The step runs
as the persistent decode chain: one launch walks the 128 linears, each waiting for its producer's
output.  The same step as 128 fused rotate_quant_linear launches (one hipGraph) is reported beside it,
and the two produce identical outputs.  ``value`` = packed-weight bytes per step / step time (GB/s).

Prefill (reported under "prefill"): LLaMA-3.1-8B-shaped layers at M = 2048, layers 0-15 W4 and
16-31 W2 MNZ; per layer 4 rotate_quant_act + 4 linears (q|k|v 6144 x 4096 and gate|up 28672 x 4096
stacked along N, o, down), replayed as one hipGraph; int8 TOPS = sum 2 M N K / step time.

Also reported: the LLaMA-2-7B-shaped stack (the same structure on those shapes), ``read_probe`` (a
plain streaming-read kernel over 2 GiB: the achievable HBM read bandwidth), ``decode_per_shape``
(each LLaMA-3.1-8B decode shape looped over >= 1 GiB of distinct weight replicas, with the read probe
over the same replicas), stacks at more tokens, the weight quantizer, KV4 attention, the level-table
linear, and the CPU oracle on the same host (``cpu_baseline``).

    python bench.py --pmc-summary FETCH.csv WRITE.csv COPY_BYTES

reads the counter files of two rocprofv3 --pmc runs of this script (FETCH_SIZE, then WRITE_SIZE, each
with --copy-probe) and writes profiles/decode_chain_cfg2_m1_traffic.json, the HBM bytes per launch of
the decode chain that the ``roofline`` of later runs reports while the kernel's sources are unchanged.

Where a linear runs on the codes of a separate rotate_quant_act call, it is given the per-token code
sums that call produced (the _ex form of the linear); without them the kernels add up the codes
themselves.

All inputs are seeded synthetic data resident in HBM before timing starts.
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

METRIC = "W2A4 linear packed-weight GB/s (% HBM peak) at M=1; int8 TOPS at M=2048"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5000.0        # MI355X dense int8 MFMA, TOPS
CHAIN_KERNEL = "k_decode_chain<0>"                   # MNZ persistent decode chain
DECODE_KERNEL_FUSED = "k_fused_decode<0, *, *, *>"   # MNZ decode kernel with the fused rotation
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_chain_cfg2_m1_traffic.json")


def _stage(name: str) -> None:
    """Progress marker on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {name}", file=sys.stderr, flush=True)


# the files the MNZ decode chain is compiled and launched from
CHAIN_SOURCES = ("qift_api.hip", "qift_chain.h", "qift_chain_mnz.hip", "qift_fwht.h", "qift_internal.h",
                 "qift_mma.h")


def _sources_hash() -> str:
    """Digest of the decode chain's sources: a committed traffic record is used only while it matches."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_02823_amd", "csrc")
    for f in CHAIN_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def _environment(torch):
    """GPU, target, ROCm/HIP and torch versions, and the clocks rocm-smi reports (a child process)."""
    props = torch.cuda.get_device_properties(0)
    env = {"gpu": torch.cuda.get_device_name(0), "arch": getattr(props, "gcnArchName", None),
           "hip": torch.version.hip, "torch": torch.__version__, "cus": props.multi_processor_count}
    if any(k.startswith("ROCPROF") for k in os.environ):
        # under the profiler every child process initialises the GPU first, and rocm-smi (a Python
        # script started through env) would then replace itself: not queried in profiled runs
        env["clocks"] = "not queried under the profiler"
        return env
    try:
        import subprocess
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=20)
        env["clocks"] = [ln.strip() for ln in r.stdout.splitlines() if "clk" in ln.lower() and "(" in ln][:8]
    except Exception as e:   # the tool may be missing; the bench line does not depend on it
        env["clocks"] = f"unavailable: {type(e).__name__}"
    return env


def _traffic_record():
    """HBM bytes per launch of the decode chain from the committed rocprofv3 PMC summary.

    Returns None unless the summary was taken on the current kernel sources.
    """
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("sources_sha") != _sources_hash():
        return None
    return rec.get("bytes_per_launch")


def _stack_plan(c):
    """(name, N, K, block, input link within the layer: -1 the previous layer's down output) of one
    layer: q|k|v and gate|up stacked along N."""
    sh = {s.name: s for s in c.linears}
    return [("qkv", sh["q"].N + sh["k"].N + sh["v"].N, sh["q"].K, sh["q"].block, -1),
            ("o", sh["o"].N, sh["o"].K, sh["o"].block, 0),
            ("gate_up", sh["gate"].N + sh["up"].N, sh["gate"].K, sh["gate"].block, 1),
            ("down", sh["down"].N, sh["down"].K, sh["down"].block, 2)]


# gain of one linear on the activations' RMS per unit s_w sqrt(K) (|y| ~ s_w s_x sqrt(K E l^2 E q^2)):
# with s_w = jitter / (gain sqrt(K)) the magnitudes stay about constant through the 32 layers
STACK_GAIN = 1.7


class DepStack:
    """32 distinct seeded MNZ layers of a LLaMA-shaped config at M = 1 with real data dependencies
    (each linear's input is a slice of an earlier linear's output), as the persistent decode chain
    (one launch) and as one fused rotate_quant_linear launch per linear."""

    def __init__(self, torch, qift, synth, cfg=2, layers=32, M=1):
        self.torch, self.qift, self.synth = torch, qift, synth
        self.cfg, self.layers, self.M = cfg, layers, M
        self.c = synth.CONFIGS[cfg]
        self.plan = _stack_plan(self.c)
        names = {1: "LLaMA-2-7B (q,k,v,o 4096x4096; gate,up 11008x4096; down 4096x11008, Hadamard 4096 / "
                    "172x64)",
                 2: "LLaMA-3.1-8B (q,o 4096x4096; k,v 1024x4096; gate,up 14336x4096; down 4096x14336, "
                    "Hadamard 4096 / 7x2048)"}
        self.workload = (f"{names[cfg]}-shaped decode stack, MNZ W2, M={M}, {layers} distinct seeded layers; "
                         "q|k|v and gate|up stacked along N; each linear reads an earlier linear's output "
                         "(o: q part of q|k|v; gate|up: o; down: gate part of gate|up; next q|k|v: down)")

    def setup(self):
        torch, qift, synth = self.torch, self.qift, self.synth
        import numpy as np
        dev = torch.device("cuda")
        self.links, self.weights = [], []
        for layer in range(self.layers):
            base = len(self.links)
            for slot, (name, N, K, b, src) in enumerate(self.plan):
                lev = synth.draw_levels_torch(qift.W2_MNZ, N, K, seed=1_000_003 * layer + 31 * self.cfg + slot,
                                              device=dev)
                jit = synth.draw_scales(qift.W2_MNZ, N, cfg=self.cfg, layer=layer, slot=slot).astype(np.float64)
                sw = (jit / np.median(jit) / (STACK_GAIN * np.sqrt(K))).astype(np.float16)
                w = qift.pack_w2(lev, torch.from_numpy(sw).to(dev), qift.W2_MNZ)
                del lev
                in_link = (base - 1 if layer else -1) if src < 0 else base + src
                self.weights.append(w)
                self.links.append(qift.ChainLink(w, b, in_link, 0))
        K0 = self.plan[0][2]
        self.x0 = torch.from_numpy(synth.config_activations(self.c, 0, 0, self.M, K0)).to(dev)
        self.outs = [torch.empty((self.M, l.w.N), dtype=torch.float16, device=dev) for l in self.links]
        self.chain = qift.Chain(self.links, self.M)
        torch.cuda.synchronize()
        self.packed_bytes = sum(w.nbytes for w in self.weights)
        # algorithmic bytes of one linear: packed words + fp16 scales + its fp16 input + fp16 output
        M = self.M
        self.alg_bytes = [l.w.N * l.w.K // 4 + 2 * l.w.N + 2 * M * l.w.K + 2 * M * l.w.N for l in self.links]

    def step_chain(self):
        """One token through the stack: the persistent decode chain (one kernel launch)."""
        self.chain.run(self.x0)

    def step_launches(self):
        """One token through the stack: one fused rotate_quant_linear launch per linear."""
        qift = self.qift
        for i, l in enumerate(self.links):
            xin = self.x0 if l.in_link < 0 else self.outs[l.in_link][:, l.in_offset:l.in_offset + l.w.K]
            qift.rotate_quant_linear(l.w, xin, l.block, out=self.outs[i])

    def paths_agree(self):
        """Both paths on the same input give identical fp16 outputs at every linear."""
        torch = self.torch
        self.step_chain()
        self.step_launches()
        torch.cuda.synchronize()
        return all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(self.chain.outs, self.outs))

    @property
    def launches_per_step(self):
        return len(self.links)


def _time_events(torch, run, steps):
    """Mean seconds per call of run over `steps` calls between HIP events on the current stream."""
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(steps):
        run()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e-3 / steps


def _capture(torch, fn):
    """A hipGraph holding fn's launches (one warm call on a side stream first)."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        fn()
    g.replay()
    torch.cuda.synchronize()
    return g


class PrefillStack:
    """cfg4: LLaMA-3.1-8B shapes, M=2048, layers 0-15 W4, 16-31 W2 MNZ; q|k|v and gate|up stacked."""

    def __init__(self, torch, qift, synth, layers=32, M=2048):
        self.torch, self.qift, self.synth = torch, qift, synth
        self.layers, self.M = layers, M
        self.c = synth.CONFIGS[4]
        sh = {s.name: s for s in self.c.linears}
        # (name, N, K, block, activation site)
        self.plan = [("qkv", sh["q"].N + sh["k"].N + sh["v"].N, sh["q"].K, sh["q"].block, 0),
                     ("o", sh["o"].N, sh["o"].K, sh["o"].block, 1),
                     ("gate_up", sh["gate"].N + sh["up"].N, sh["gate"].K, sh["gate"].block, 2),
                     ("down", sh["down"].N, sh["down"].K, sh["down"].block, 3)]

    def setup(self):
        torch, qift, synth = self.torch, self.qift, self.synth
        dev = torch.device("cuda")
        self.weights = []
        for layer in range(self.layers):
            fmt = self.c.fmt_of_layer[layer]
            ws = []
            for slot, (name, N, K, b, site) in enumerate(self.plan):
                lev = synth.draw_levels_torch(fmt, N, K, seed=7_000_003 * layer + slot, device=dev)
                sc = torch.from_numpy(synth.draw_scales(fmt, N, cfg=4, layer=layer, slot=slot)).to(dev)
                ws.append(qift.pack_w4(lev, sc) if fmt == qift.W4_SYM
                          else qift.pack_w2(lev, sc, fmt))
                del lev
            self.weights.append(ws)
        # one synthetic input per activation site, shared by the layers
        self.x = [torch.from_numpy(synth.config_activations(self.c, 0, site, self.M, K)).to(dev)
                  for (_, _, K, _, site) in self.plan]
        self.acts = [qift.alloc_act(self.M, K, dev) for (_, _, K, _, _) in self.plan]
        self.outs = [torch.empty((self.M, N), dtype=torch.float16, device=dev) for (_, N, _, _, _) in self.plan]
        torch.cuda.synchronize()
        self.ops = self.layers * sum(2 * self.M * N * K for (_, N, K, _, _) in self.plan)

    def step(self):
        qift = self.qift
        for layer in range(self.layers):
            ws = self.weights[layer]
            for i, (name, N, K, b, site) in enumerate(self.plan):
                act = qift.rotate_quant_act(self.x[i], b, out=self.acts[i])
                qift.linear(ws[i], act, out=self.outs[i], use_sum=True)


class SweepStack:
    """32 distinct seeded layers of one config at M tokens: cfg2 (LLaMA-3.1-8B, MNZ; q|k|v, o, gate|up,
    down) or cfg3 (LLaMA-3.1-8B MLP, PoT; gate|up, down), every linear on a fixed synthetic input of its
    site (no dependency between linears).  M = 1 runs the fused rotate+linear entry, larger M one
    rotate_quant_act per input and the linear on its codes (the fused entry also takes M = 4, but
    measured slower there: 2.59 vs 1.58 ms for this stack, its workgroups each rotating all four
    tokens of K = 14336)."""

    def __init__(self, torch, qift, synth, cfg, M, layers=32):
        self.torch, self.qift, self.synth = torch, qift, synth
        self.cfg, self.M, self.layers = cfg, M, layers
        c = synth.CONFIGS[cfg]
        sh = {s.name: s for s in c.linears}
        self.plan = [("gate_up", sh["gate"].N + sh["up"].N, sh["gate"].K, sh["gate"].block, 2),
                     ("down", sh["down"].N, sh["down"].K, sh["down"].block, 3)]
        if "q" in sh:
            self.plan = [("qkv", sh["q"].N + sh["k"].N + sh["v"].N, sh["q"].K, sh["q"].block, 0),
                         ("o", sh["o"].N, sh["o"].K, sh["o"].block, 1)] + self.plan
        self.fmt = c.fmt_of_layer[0]
        self.fused = M == 1   # fused entry at one token; for more, one rotation per input then the linear

    def setup(self):
        torch, qift, synth = self.torch, self.qift, self.synth
        dev = torch.device("cuda")
        c = synth.CONFIGS[self.cfg]
        self.weights = []
        for layer in range(self.layers):
            ws = []
            for slot, (name, N, K, b, site) in enumerate(self.plan):
                lev = synth.draw_levels_torch(self.fmt, N, K, seed=3_000_017 * layer + 101 * self.cfg + slot,
                                              device=dev)
                sc = torch.from_numpy(synth.draw_scales(self.fmt, N, cfg=self.cfg, layer=layer, slot=slot)).to(dev)
                ws.append(qift.pack_w2(lev, sc, self.fmt))
                del lev
            self.weights.append(ws)
        self.x = [torch.from_numpy(synth.config_activations(c, 0, site, self.M, K)).to(dev)
                  for (_, _, K, _, site) in self.plan]
        self.acts = [qift.alloc_act(self.M, K, dev) for (_, _, K, _, _) in self.plan]
        self.outs = [torch.empty((self.M, N), dtype=torch.float16, device=dev) for (_, N, _, _, _) in self.plan]
        # one workspace for the linears that take one at this M (the skinny linear split over K up to 64
        # tokens, the FP4 x FP6 GEMM above)
        self.need = [qift.workspace_bytes(w, self.M) for w in self.weights[0]]
        self.ws = torch.empty(max(self.need), dtype=torch.uint8, device=dev) if max(self.need) else None
        torch.cuda.synchronize()
        self.packed_bytes = sum(w.nbytes for ws in self.weights for w in ws)
        self.ops = self.layers * sum(2 * self.M * N * K for (_, N, K, _, _) in self.plan)

    def step(self):
        qift = self.qift
        for layer in range(self.layers):
            ws = self.weights[layer]
            for i, (name, N, K, b, site) in enumerate(self.plan):
                if self.fused:
                    qift.rotate_quant_linear(ws[i], self.x[i], b, out=self.outs[i])
                else:
                    act = qift.rotate_quant_act(self.x[i], b, out=self.acts[i])
                    qift.w2a4_linear(ws[i], act, out=self.outs[i], use_sum=True,
                                     workspace=self.ws[:self.need[i]] if self.need[i] else None)


def stack_sweep(torch, qift, synth, reps=20):
    """Tokens/s and packed GB/s of the cfg2 stack at M in {1, 4, 16, 128} and the cfg3 PoT MLP stack at
    M in {1, 8, 64} (hipGraph replays, inputs resident)."""
    rows = []
    for cfg, Ms in ((2, (1, 4, 16, 128)), (3, (1, 8, 64))):
        for M in Ms:
            st = SweepStack(torch, qift, synth, cfg, M)
            st.setup()
            st.step()
            torch.cuda.synchronize()
            dt = _time_graph(torch, st.step, reps)
            gbs = st.packed_bytes / dt / 1e9
            c = synth.CONFIGS[cfg]
            rows.append({"config": c.label, "M": M, "layers": st.layers,
                         "linears": "+".join(n for n, *_ in st.plan),
                         "path": "fused rotate_quant_linear" if st.fused else "rotate_quant_act + w2a4_linear",
                         "ms_per_step": round(dt * 1e3, 4), "tokens_per_s": round(M / dt, 1),
                         "packed_GBs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                         "int8_tops": round(st.ops / dt / 1e12, 2)})
            st = None
            torch.cuda.empty_cache()
    return rows


def _time_graph(torch, fn, reps):
    """Mean seconds per replay of a graph holding fn's launches (one warm replay first)."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        fn()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    del g
    return a.elapsed_time(b) * 1e-3 / reps


def read_probe(torch, qift, nbytes=1 << 31, reps=10):
    """Achievable HBM read bandwidth: the streaming-read probe over one large buffer."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    parts = torch.empty(qift.read_probe_slots(nbytes), dtype=torch.int32, device="cuda")
    dt = _time_graph(torch, lambda: qift.hbm_read_probe(buf, parts), reps)
    del buf
    return {"bytes": nbytes, "GBs": round(nbytes / dt / 1e9, 1), "pct_hbm_peak": round(100 * nbytes / dt / 1e9 / HBM_PEAK_GBS, 1)}


def decode_per_shape(torch, qift, synth, min_bytes=1 << 30, reps=10):
    """Each LLaMA-3.1-8B decode shape's kernel looped over >= min_bytes of distinct weight replicas
    (M = 1): fused rotate+linear, the linear on precomputed codes, and the read probe over the same
    replicas (the floor for that launch size)."""
    c = synth.CONFIGS[2]
    plan = [(name, N, K, b, site) for site, (name, N, K, b, _) in enumerate(_stack_plan(c))]
    rows = []
    for name, N, K, b, site in plan:
        dev = torch.device("cuda")
        lev = synth.draw_levels_torch(qift.W2_MNZ, N, K, seed=99 + site, device=dev)
        sc = torch.from_numpy(synth.draw_scales(qift.W2_MNZ, N, cfg=2, layer=0, slot=site)).to(dev)
        base = qift.pack_w2(lev, sc, qift.W2_MNZ)
        del lev
        R = -(-min_bytes // base.nbytes)
        reps_w = [qift.Packed(base.fmt, N, K, base.words.clone(), sc) for _ in range(R)]
        x = torch.from_numpy(synth.config_activations(c, 0, site, 1, K)).to(dev)
        act = qift.rotate_quant_act(x, b)
        y = torch.empty((1, N), dtype=torch.float16, device=dev)
        parts = torch.empty(qift.read_probe_slots(base.nbytes), dtype=torch.int32, device=dev)
        total = R * base.nbytes

        def fused():
            for w in reps_w:
                qift.rotate_quant_linear(w, x, b, out=y)

        def lin():
            for w in reps_w:
                qift.w2a4_linear(w, act, out=y, use_sum=True)

        def probe():
            for w in reps_w:
                qift.hbm_read_probe(w.words, parts)

        t_f, t_l, t_p = (_time_graph(torch, f, reps) for f in (fused, lin, probe))
        gbs = lambda t: round(total / t / 1e9, 1)
        rows.append({"linear": name, "N": N, "K": K, "packed_bytes": base.nbytes, "replicas": R,
                     "fused_GBs": gbs(t_f), "fused_us": round(t_f / R * 1e6, 2),
                     "linear_on_act_q_GBs": gbs(t_l), "linear_on_act_q_us": round(t_l / R * 1e6, 2),
                     "read_probe_GBs": gbs(t_p), "read_probe_us": round(t_p / R * 1e6, 2),
                     "fused_pct_hbm_peak": round(100 * total / t_f / 1e9 / HBM_PEAK_GBS, 1),
                     "fused_pct_of_read_probe": round(100 * t_p / t_f, 1)})
        del reps_w, base
        torch.cuda.empty_cache()
    return rows


# the reference grids of Sec. 3.3: Lloyd-Max (Eq. (9)) and NF2 (Eq. (10))
LLOYD_GRID = (-1.5104, -0.4528, 0.4528, 1.5104)
NF2_GRID = (-1.0, -0.2525685, 0.2525685, 1.0)


def lut_decode(torch, qift, synth, min_bytes=1 << 29, reps=10):
    """The level-table linear (W2_LUT: the Lloyd-Max and NF2 reference grids) at the cfg1 decode
    shapes, M = 1 on precomputed activation codes, looped over >= min_bytes of distinct code
    replicas; the integer MNZ linear on the same replicas beside it."""
    c = synth.CONFIGS[1]
    sh = {s.name: s for s in c.linears}
    plan = [("q,k,v", 3 * sh["q"].N, sh["q"].K, sh["q"].block, 0), ("o", sh["o"].N, sh["o"].K, sh["o"].block, 1),
            ("gate,up", 2 * sh["gate"].N, sh["gate"].K, sh["gate"].block, 2),
            ("down", sh["down"].N, sh["down"].K, sh["down"].block, 3)]
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    rows = []
    for name, N, K, b, site in plan:
        codes = torch.randint(0, 4, (N, K), dtype=torch.int8, device=dev, generator=gen)
        sc = torch.from_numpy(synth.draw_scales(qift.W2_MNZ, N, cfg=1, layer=0, slot=site)).to(dev)
        base = qift.pack_w2(codes, sc, qift.W2_LUT)
        del codes
        R = -(-min_bytes // base.nbytes)
        reps_w = [qift.Packed(qift.W2_LUT, N, K, base.words.clone(), sc) for _ in range(R)]
        reps_i = [qift.Packed(qift.W2_MNZ, N, K, w.words, sc) for w in reps_w]
        x = torch.from_numpy(synth.config_activations(c, 0, site, 1, K)).to(dev)
        act = qift.rotate_quant_act(x, b)
        y = torch.empty((1, N), dtype=torch.float16, device=dev)
        total = R * base.nbytes
        row = {"linear": name, "N": N, "K": K, "packed_bytes": base.nbytes, "replicas": R}
        for gname, grid in (("lloyd", LLOYD_GRID), ("nf2", NF2_GRID)):
            def run(grid=grid):
                for w in reps_w:
                    qift.w2a4_lut_linear(w, grid, act, out=y)
            t = _time_graph(torch, run, reps)
            row[gname + "_us"] = round(t / R * 1e6, 2)
            row[gname + "_GBs"] = round(total / t / 1e9, 1)

        def mnz():
            for w in reps_i:
                qift.w2a4_linear(w, act, out=y, use_sum=True)
        t = _time_graph(torch, mnz, reps)
        row["mnz_integer_us"] = round(t / R * 1e6, 2)
        rows.append(row)
        del reps_w, reps_i, base
        torch.cuda.empty_cache()
    return {"workload": "LLaMA-2-7B-shaped decode linears (cfg1), M = 1, activation codes precomputed; "
                        "random 2-bit codes (the kernel's work does not depend on them)", "rows": rows}


FP64_VECTOR_PEAK_TFLOPS = 78.6
# per candidate and weight, fp64: the threshold test fma(-2.5, s, |w|) (2 flops), s * level, w - s * level,
# d * d and the add into the error sum (the scale search's inner loop; there is no division in it)
POT_FLOPS_PER_WEIGHT = 64 * 6


def weight_quantizer(torch, qift, synth, reps=5):
    """The GPU weight quantizer on one LLaMA-3.1-8B layer (its 7 linears, 218M fp32 weights) per
    format: rotation, per-row scale and levels (the offline step before packing; hipGraph replays,
    weights resident).  MNZ and W4 move 4 B in + 1 B out per weight (HBM roofline); the PoT scale
    search is fp64 arithmetic, priced at 6 flops per candidate and weight against the fp64 vector
    peak."""
    c = synth.CONFIGS[2]
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(2)
    mats = []
    for s in c.linears:
        # 0.02 * Student-t(5): z / sqrt(chi2_5 / 5)
        z = torch.randn((s.N, s.K), device=dev, generator=gen)
        chi = torch.zeros_like(z)
        for _ in range(5):
            chi.add_(torch.randn((s.N, s.K), device=dev, generator=gen).square_())
        W = (0.02 * z / torch.sqrt(chi / 5.0)).contiguous()
        del z, chi
        mats.append((W, s.block, torch.empty((s.N, s.K), dtype=torch.int8, device=dev),
                     torch.empty(s.N, dtype=torch.float16, device=dev)))
    weights = sum(W.numel() for W, *_ in mats)
    rows = sum(W.shape[0] for W, *_ in mats)
    out = {"workload": "one LLaMA-3.1-8B layer: q, k, v, o, gate, up, down (218,103,808 fp32 weights; "
                       "4096 blocks for K 4096, 7 blocks of 2048 for K 14336)"}
    for fmt, name in ((qift.W2_MNZ, "W2 MNZ (RMS)"), (qift.W2_POT, "W2 PoT (64-candidate MSE)"),
                      (qift.W4_SYM, "W4 (absmax/7)")):
        def layer():
            for W, b, L, S in mats:
                qift.quantize_weights(W, b, fmt, levels=L, scales=S)
        dt = _time_graph(torch, layer, reps)
        gbs = (5 * weights + 2 * rows) / dt / 1e9
        rec = {"ms_per_layer": round(dt * 1e3, 3), "gweights_per_s": round(weights / dt / 1e9, 2),
               "GBs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2)}
        if fmt == qift.W2_POT:
            tf = POT_FLOPS_PER_WEIGHT * weights / dt / 1e12
            rec["roofline"] = {"bound": "alu", "achieved": round(tf, 2), "peak": FP64_VECTOR_PEAK_TFLOPS,
                               "unit": "TFLOP/s", "frac": round(tf / FP64_VECTOR_PEAK_TFLOPS, 4)}
        else:
            rec["roofline"] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                               "frac": round(gbs / HBM_PEAK_GBS, 4)}
        out[name] = rec
    del mats
    return out


def kv4_attention(torch, qift, reps=10, layers=32):
    """KV4 caches of the 32 layers of LLaMA-3.1-8B (32 query heads, 8 KV heads, head_dim 128): one
    decode step's attention over T cached tokens for B sequences, i.e. 32 launches over 32 distinct
    caches in one hipGraph (HBM roofline: each 4-bit cache is read once, 64 B of codes + 4 B scale
    + 1 B zero-point per token, KV head and tensor), for both cache row orders (head-major
    [B, Hkv, T], token-major [B, T, Hkv]); and the quantizer writing one layer's cache of T tokens
    (fp16 in, KV4 out)."""
    dev = torch.device("cuda")
    Hq, Hkv = 32, 8
    gen = torch.Generator(device=dev)
    gen.manual_seed(4)
    rows = []
    for B, T in ((1, 4096), (1, 32768), (16, 4096)):
        for head_major in (True, False):
            shape = (B, Hkv, T, 128) if head_major else (B, T, Hkv, 128)
            caches = []
            for _ in range(layers):
                K = torch.randn(shape, device=dev, generator=gen).half()
                V = torch.randn(shape, device=dev, generator=gen).half()
                caches.append((qift.kv4_quant(K), qift.kv4_quant(V)))
            q = torch.randn((B, Hq, 128), device=dev, generator=gen).half()
            y = torch.empty((B, Hq, 128), dtype=torch.float16, device=dev)
            ws = torch.empty(qift.lib().qift_kv4_attention_workspace_bytes(B, Hq, Hkv, 128, T), dtype=torch.uint8,
                             device=dev)

            def step():
                for k, v in caches:
                    qift.kv4_attention_decode(q, k, v, out=y, workspace=ws, head_major=head_major)
            dt = _time_graph(torch, step, reps) / layers
            cache = 2 * B * T * Hkv * (64 + 4 + 1)
            gbs = (cache + 4 * B * Hq * 128) / dt / 1e9
            row = {"B": B, "T": T, "layout": "head-major" if head_major else "token-major",
                   "attention_us_per_layer": round(dt * 1e6, 2), "cache_bytes_per_layer": cache,
                   "attention_GBs": round(gbs, 1), "attention_pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2)}
            if head_major:
                k, v = caches[0]

                def quant():
                    for _ in range(4):
                        qift.kv4_quant(K, out=k)
                        qift.kv4_quant(V, out=v)
                dq = _time_graph(torch, quant, reps) / 4
                row["quant_us_per_layer"] = round(dq * 1e6, 2)
                row["quant_GBs"] = round((2 * B * T * Hkv * 256 + cache) / dq / 1e9, 1)
            rows.append(row)
            del K, V, caches, ws
            torch.cuda.empty_cache()
    return {"workload": "LLaMA-3.1-8B attention at decode, 32 layers: Hq 32, Hkv 8, head_dim 128, KV4 cache "
                        "(clip 0.95), T cached tokens per sequence, B sequences", "rows": rows}


def _median(fn, runs):
    """Median seconds of `runs` calls of fn (and every time, ascending)."""
    ts = []
    for _ in range(runs):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    ts.sort()
    return ts[len(ts) // 2], ts


def cpu_baseline(synth, runs=3):
    """The oracle as it stands (fp64 numpy; its integer dot is an fp64 BLAS matmul of the integer-valued
    operands, exact since every partial sum stays below 2^53), timed on this host's cores.

    value: one LLaMA-3.1-8B decode layer (q, k, v, o, gate, up, down; MNZ; 4 activation quantizations)
    at M = 1, all BLAS threads, median of `runs` passes, as packed-weight GB/s (the headline's unit;
    32 layers take 32 times as long).  detail (one pass each): the same layer on one thread; the tiny
    config in full (weights -> rotation -> quantization -> packing, activation quantization, linear,
    median of 5); one PoT MLP layer (gate, up, down) at M 1, 8 and 64; one linear of each
    LLaMA-3.1-8B shape at M = 2048 in W4 and in W2 MNZ (all threads; the int4 activation codes there
    are seeded draws, since the linear's time does not depend on their values, and the activation
    quantization is timed apart on 256 tokens), and one of them on one thread.  Each distinct
    (format, N, K) is drawn and packed once."""
    import numpy as np
    from oracle import hadamard, levels as olev, linear as olin, pack as opack, quant
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    t_start = time.perf_counter()
    packs = {}

    def packed(fmt, N, K, cfg):
        key = (fmt, N, K)
        if key not in packs:
            L = synth.draw_levels(fmt, N, K, cfg=cfg, layer=0, slot=len(packs))
            packs[key] = (opack.pack(L, fmt), synth.draw_scales(fmt, N, cfg=cfg, layer=0, slot=len(packs)))
        return packs[key]

    def layer_fn(cfg, fmt, names, M):
        c = synth.CONFIGS[cfg]
        sh = {s.name: s for s in c.linears}
        prepared = [(sh[nm],) + packed(fmt, sh[nm].N, sh[nm].K, cfg) for nm in names]
        sites = {}
        for s, _, _ in prepared:
            site = synth.SITE_OF[s.name]
            sites.setdefault(site, (synth.config_activations(c, 0, site, M, s.K), s.block))

        def run():
            qa = {site: quant.act_quant(x, b) for site, (x, b) in sites.items()}
            for s, P, sw in prepared:
                q, sx, _, _ = qa[synth.SITE_OF[s.name]]
                olin.linear(P, sw, fmt, s.K, q, sx)
        return run, sum(P.nbytes for _, P, _ in prepared)

    # ---- the headline's unit: one cfg2 decode layer at M = 1
    run2, packed2 = layer_fn(2, olev.FMT_W2_MNZ, synth.LINEARS, 1)
    run2()   # warm the oracle's cached Hadamard matrices
    t_all, ts_all = _median(run2, runs)
    with threadpool_limits(1):
        t_one, _ = _median(run2, 1)
    detail = {"cfg2_layer_M1": {"packed_bytes": packed2, "all_threads_s": [round(t, 3) for t in ts_all],
                                "one_thread_s": round(t_one, 3), "one_thread_GBs": round(packed2 / t_one / 1e9, 4),
                                "tokens_per_s_32_layers": round(1.0 / (32 * t_all), 4)}}

    # ---- the tiny config in full
    c0 = synth.CONFIGS[0]
    s0 = c0.linears[0]

    def tiny():
        W = synth.weights_fp32(0, 0, "lin", s0.N, s0.K)
        L, s_w = quant.quantize_mnz_rms(hadamard.rotate_weights(W, s0.block))
        P = opack.pack(L, olev.FMT_W2_MNZ)
        x = synth.config_activations(c0, 0, 0, c0.Ms[0], s0.K)
        q, sx, _, _ = quant.act_quant(x, s0.block)
        olin.linear(P, s_w, olev.FMT_W2_MNZ, s0.K, q, sx)
    tiny()
    t0_, _ = _median(tiny, 5)
    detail["cfg0_full"] = {"median_s": round(t0_, 5), "runs": 5,
                           "what": f"{c0.Ms[0]}x{s0.N}x{s0.K}: weights, rotation, RMS levels, packing, "
                                   "activation quantization, linear"}

    # ---- one PoT MLP layer at M 1, 8, 64
    rows3 = []
    for M in (1, 8, 64):
        run3, packed3 = layer_fn(3, olev.FMT_W2_POT, ("gate", "up", "down"), M)
        t, _ = _median(run3, 1)
        rows3.append({"M": M, "s": round(t, 3), "packed_GBs": round(packed3 / t / 1e9, 4)})
    detail["cfg3_layer"] = rows3

    # ---- one linear per LLaMA-3.1-8B shape at M = 2048 (W4 and W2 MNZ)
    c4 = synth.CONFIGS[4]
    sh4 = {s.name: s for s in c4.linears}
    M4 = 2048
    gen = np.random.default_rng(7)
    rows4 = []
    qs = {}
    for nm in ("q", "k", "gate", "down"):
        s = sh4[nm]
        if s.K not in qs:
            x = synth.config_activations(c4, 0, synth.SITE_OF[nm], 256, s.K)
            a0 = time.perf_counter()
            quant.act_quant(x, s.block)
            rows4.append({"act_quant": f"256 tokens x {s.K}, block {s.block}", "s": round(time.perf_counter() - a0, 3)})
            qs[s.K] = (gen.integers(-7, 8, size=(M4, s.K)).astype(np.int8), np.full(M4, 0.01, np.float32))
        q, sx = qs[s.K]
        for fmt, fname in ((olev.FMT_W4_SYM, "W4"), (olev.FMT_W2_MNZ, "W2 MNZ")):
            P, sw = packed(fmt, s.N, s.K, 4)
            t, _ = _median(lambda: olin.linear(P, sw, fmt, s.K, q, sx), 1)
            rows4.append({"linear": nm, "format": fname, "N": s.N, "K": s.K, "s": round(t, 3),
                          "int8_equiv_TOPS": round(2 * M4 * s.N * s.K / t / 1e12, 4)})
    s = sh4["q"]
    P, sw = packed(olev.FMT_W4_SYM, s.N, s.K, 4)
    q, sx = qs[s.K]
    with threadpool_limits(1):
        t, _ = _median(lambda: olin.linear(P, sw, olev.FMT_W4_SYM, s.K, q, sx), 1)
    rows4.append({"linear": "q", "format": "W4", "threads": 1, "s": round(t, 3),
                  "int8_equiv_TOPS": round(2 * M4 * s.N * s.K / t / 1e12, 4)})
    detail["cfg4_linears_M2048"] = rows4
    try:
        with open("/proc/cpuinfo") as f:
            detail["cpu_model"] = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:  # pragma: no cover
        detail["cpu_model"] = None
    detail["total_s"] = round(time.perf_counter() - t_start, 1)
    return {"value": round(packed2 / t_all / 1e9, 4), "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one LLaMA-3.1-8B decode layer (7 MNZ linears, 4 activation quantizations) at M=1, "
                      f"median of {runs} passes after one warm-up ({t_all:.2f} s each; {packed2} packed bytes "
                      f"per pass, 1/32 of the decode step); host has {os.cpu_count()} logical CPUs",
            "detail": detail}


def dep_stack_record(torch, qift, synth, cfg, steps, warmup, layers=32):
    """Chain and per-launch timings of one DepStack (hipGraph replays), and whether they agree."""
    st = DepStack(torch, qift, synth, cfg=cfg, layers=layers)
    st.setup()
    agree = st.paths_agree()
    rec = {"workload": st.workload, "packed_bytes_per_step": st.packed_bytes, "paths_agree": agree}
    for name, fn in (("chain", st.step_chain), ("launches", st.step_launches)):
        g = _capture(torch, fn)
        for _ in range(warmup):
            g.replay()
        dt = _time_events(torch, g.replay, steps)
        rec[name] = {"ms_per_step": round(dt * 1e3, 4), "tokens_per_s": round(st.M / dt, 1),
                     "packed_GBs": round(st.packed_bytes / dt / 1e9, 1),
                     "pct_hbm_peak": round(100 * st.packed_bytes / dt / 1e9 / HBM_PEAK_GBS, 2)}
        del g
    st = None
    torch.cuda.empty_cache()
    return rec


def pmc_summary(fetch_csv, write_csv, copy_bytes):
    """Traffic record of the decode chain from two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE, in KiB
    per dispatch) of this script with --copy-probe: each counter is scaled by what it reads for the
    1 GiB device copies of the same run (copy_bytes read and written per copy)."""
    import csv

    def per_kernel(path, counter):
        vals = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return vals

    f, w = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    pick = lambda d, key: next(v for k, v in d.items() if key(k))
    is_chain = lambda k: "k_decode_chain<0>" in k
    is_copy = lambda k: "copybuffer" in k.lower()   # the runtime's device-to-device copy kernel
    # the four 1 GiB copies of --copy-probe: the largest copy dispatches of each run
    copy_f = sorted(v for k, vs in f.items() if is_copy(k) for v in vs)[-4:]
    copy_w = sorted(v for k, vs in w.items() if is_copy(k) for v in vs)[-4:]
    ff = copy_bytes / (sum(copy_f) / len(copy_f))
    wf = copy_bytes / (sum(copy_w) / len(copy_w))
    cf, cw = pick(f, is_chain), pick(w, is_chain)
    fetch = sum(cf) / len(cf) * ff
    write = sum(cw) / len(cw) * wf
    rec = {"kernel": CHAIN_KERNEL + " (MNZ, M=1, LLaMA-3.1-8B 32-layer decode step)",
           "sources_sha": _sources_hash(), "bytes_per_launch": int(fetch + write),
           "fetch_bytes_per_launch": int(fetch), "write_bytes_per_launch": int(write),
           "fetch_factor": round(ff, 4), "write_factor": round(wf, 4),
           "dispatches": {"fetch": len(cf), "write": len(cw), "copy": len(copy_f)}}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--prefill-steps", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-cfg1", action="store_true", help="skip the LLaMA-2-7B-shaped stack")
    ap.add_argument("--no-per-shape", action="store_true",
                    help="skip the per-shape replica loops and the read probe")
    ap.add_argument("--no-wquant", action="store_true", help="skip the weight quantizer timing")
    ap.add_argument("--no-kv4", action="store_true", help="skip the KV4 attention timing")
    ap.add_argument("--no-lut", action="store_true", help="skip the level-table linear timing")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the cfg2 (M 1/4/16/128) and cfg3 PoT (M 1/8/64) stack sweep")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run 1 GiB device copies (HBM byte-counter calibration under rocprofv3)")
    ap.add_argument("--pmc-summary", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_BYTES"),
                    help="write the decode chain's traffic record from two rocprofv3 --pmc runs and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], float(args.pmc_summary[2]))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the quantized linear shards by output rows with no "
              "exchange, so the job throughput is the per-GPU figure; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_02823_amd import qift, synth
    qift.lib()
    torch.cuda.set_device(0)

    # ---------------------------------------------------------------- decode (headline)
    _stage("decode step (LLaMA-3.1-8B stack, persistent chain)")
    dec = DepStack(torch, qift, synth, cfg=2, layers=args.layers, M=1)
    dec.setup()
    agree = dec.paths_agree()
    if qift.device_error(clear=True):
        raise RuntimeError("a wait of the decode chain gave up")
    graph = _capture(torch, dec.step_chain)
    run = graph.replay
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record()
    for _ in range(args.steps):
        run()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = t0.elapsed_time(t1) / args.steps
    gbs = dec.packed_bytes / (ms * 1e-3) / 1e9
    dev_err = qift.device_error(clear=True)
    # the distribution of single steps (each replay between its own events), after the timed region
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ev:
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    one = sorted(a.elapsed_time(b) for a, b in ev)
    pct = lambda f: one[min(len(one) - 1, int(round(f * (len(one) - 1))))]
    step_dist = {"median_ms": round(pct(0.5), 4), "p10_ms": round(pct(0.1), 4), "p90_ms": round(pct(0.9), 4),
                 "single_steps": len(one)}
    # the dominant kernel is the chain itself, one launch per step: its average launch duration is the
    # timed region's event time per step (the graph holds just that launch, on this stream)
    avg_dur = ms * 1e-3
    alg = sum(dec.alg_bytes)
    achieved = alg / avg_dur / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": _traffic_record(),
                "kernel": CHAIN_KERNEL, "avg_launch_us": round(avg_dur * 1e6, 2), "alg_bytes_per_launch": int(alg)}
    del graph

    # the same step as one fused launch per linear (hipGraph), for comparison
    _stage("decode step as per-linear launches")
    lgraph = _capture(torch, dec.step_launches)
    for _ in range(args.warmup):
        lgraph.replay()
    lt = _time_events(torch, lgraph.replay, args.steps)
    del lgraph
    launches = {"ms_per_step": round(lt * 1e3, 4), "packed_GBs": round(dec.packed_bytes / lt / 1e9, 1),
                "pct_hbm_peak": round(100 * dec.packed_bytes / lt / 1e9 / HBM_PEAK_GBS, 2),
                "tokens_per_s": round(dec.M / lt, 1), "launches_per_step": dec.launches_per_step,
                "us_per_launch": round(lt / dec.launches_per_step * 1e6, 3), "kernel": DECODE_KERNEL_FUSED}

    out = {"metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "i8xi2->i32", "data": "synthetic",
           "config": {"workload": dec.workload, "tokens_per_step": dec.M, "layers": dec.layers,
                      "linears_per_step": dec.launches_per_step, "packed_bytes_per_step": dec.packed_bytes,
                      "launch": "persistent decode chain (one kernel per step), hipGraph replays",
                      "rotation": "fused into each linear"},
           "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
           "tokens_per_s": round(dec.M / (ms * 1e-3), 1),
           "host_wall_s": round(wall, 3),
           "step_ms_distribution": step_dist,
           "paths_agree": agree, "device_error_bits": dev_err,
           "decode_launches": launches,
           "roofline": roofline,
           "env": _environment(torch)}
    dec = None
    torch.cuda.empty_cache()

    if not args.no_cfg1:
        _stage("LLaMA-2-7B-shaped stack")
        out["cfg1_stack"] = dep_stack_record(torch, qift, synth, 1, min(args.steps, 20), args.warmup, args.layers)

    # ---------------------------------------------------------------- per-shape loops, read probe
    if not args.no_per_shape:
        _stage("read probe and per-shape decode loops")
        out["read_probe"] = read_probe(torch, qift)
        out["decode_per_shape"] = decode_per_shape(torch, qift, synth)
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- cfg2 / cfg3 stacks at several M
    if not args.no_sweep:
        _stage("stack sweep")
        out["stack_sweep"] = stack_sweep(torch, qift, synth)
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- offline weight quantizer
    if not args.no_wquant:
        _stage("weight quantizer")
        out["weight_quantizer"] = weight_quantizer(torch, qift, synth)
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- KV4 cache and decode attention
    if not args.no_kv4:
        _stage("KV4 attention")
        out["kv4_attention"] = kv4_attention(torch, qift)
        torch.cuda.empty_cache()

    if not args.no_lut:
        _stage("level-table linear")
        out["lut_decode"] = lut_decode(torch, qift, synth)
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- prefill
    if not args.no_prefill:
        _stage("prefill")
        pre = PrefillStack(torch, qift, synth, layers=args.layers)
        pre.setup()
        pgraph = _capture(torch, pre.step)
        pms = _time_events(torch, pgraph.replay, args.prefill_steps) * 1e3
        del pgraph
        tops = pre.ops / (pms * 1e-3) / 1e12
        # per linear shape and weight format: one layer's launch of each, replayed in a graph
        per_shape = []
        for layer in sorted({0, args.layers - 1}):
            fname = "W4" if pre.c.fmt_of_layer[layer] == qift.W4_SYM else "W2 MNZ"
            for i, (name, N, K, blk, site) in enumerate(pre.plan):
                w = pre.weights[layer][i]
                qift.rotate_quant_act(pre.x[i], blk, out=pre.acts[i])
                ops = 2 * pre.M * N * K
                # the int8 MFMA kernel; for MNZ also the FP4 x FP6 scaled-MFMA kernel (its workspace
                # selects it; the FP6 re-coding of the activations is inside the timed call)
                variants = [("int8 MFMA", None)]
                if qift.workspace_bytes(w, pre.M):
                    variants.append(("FP4 x FP6 MFMA", torch.empty(qift.workspace_bytes(w, pre.M),
                                                                   dtype=torch.uint8, device="cuda")))
                for path, ws in variants:
                    dt = _time_graph(torch, lambda: qift.linear(w, pre.acts[i], out=pre.outs[i], workspace=ws, use_sum=True), 10)
                    per_shape.append({"linear": name, "format": fname, "path": path, "N": N, "K": K,
                                      "us": round(dt * 1e6, 2), "int8_tops": round(ops / dt / 1e12, 2),
                                      "pct_int8_peak": round(100 * ops / dt / 1e12 / INT8_PEAK_TOPS, 2)})
        out["prefill"] = {"workload": "LLaMA-3.1-8B-shaped prefill, M=2048, layers 0-15 W4 / 16-31 W2 MNZ, "
                                      "4 rotate_quant_act + 4 linears per layer (q|k|v and gate|up stacked "
                                      "along N), one hipGraph",
                          "ms_per_step": round(pms, 3), "int8_tops": round(tops, 2),
                          "pct_int8_peak": round(100 * tops / INT8_PEAK_TOPS, 2),
                          "steps": args.prefill_steps, "per_shape": per_shape}
        pre = None
        torch.cuda.empty_cache()

    if args.copy_probe:
        _stage("copy probe")
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---------------------------------------------------------------- CPU oracle baseline
    if not args.no_cpu:
        _stage("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(synth)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
