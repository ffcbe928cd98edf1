"""Throughput of the rotated W2A4 quantized linear on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-prefill] [--no-cpu]

Decode (the headline ``value``): LLaMA-2-7B-shaped layers (q,k,v,o 4096x4096;
gate,up 11008x4096; down 4096x11008 with 172 Hadamard blocks of 64), MNZ
2-bit weights, M = 1 token.  A step pushes one token through 32 distinct
seeded layers (1.62 GB of packed words, the depth of LLaMA-2-7B) so that the
weights stream from HBM rather than the 256 MB Infinity Cache.  Per layer: 4
rotate_quant_linear launches (q|k|v, o, gate|up, down; q|k|v and gate|up are
stacked along N since they share their input), each rotating and quantizing
its fp16 input inside the kernel; with --unfused, 4 rotate_quant_act + 4
w2a4_linear launches instead.  The step is captured once as a hipGraph and
replayed.
``value`` = packed-weight bytes per step / step time (GB/s).

Prefill (reported under "prefill"): LLaMA-3.1-8B-shaped layers at M = 2048,
layers 0-15 W4 and 16-31 W2 MNZ; per layer 4 rotate_quant_act + 4 linears
(q|k|v 6144 x 4096 and gate|up 28672 x 4096 stacked along N, o, down);
int8 TOPS = sum 2 M N K / step time.

Also reported (measurement helpers): ``read_probe`` = the achievable HBM read
bandwidth (a plain streaming-read kernel over 2 GiB); ``decode_per_shape`` =
each decode shape's kernel looped over >= 1 GiB of distinct weight replicas
(fused kernel, linear on precomputed act_q, and the read probe over the same
replicas, i.e. the floor for that launch size); ``stack_kernel_sum_ms`` = the
decode step's kernels back to back.

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
DECODE_KERNEL_FUSED = "k_fused_decode<0, *, *, *>"   # MNZ decode kernel with the fused rotation
DECODE_KERNEL = "k_decode_deep<0, 1, 1, *>"          # MNZ decode kernel on staged act_q


def _stage(name: str) -> None:
    """Progress marker on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {name}", file=sys.stderr, flush=True)


# the files the MNZ decode kernel is compiled and launched from
DECODE_SOURCES = ("qift_api.hip", "qift_fused.h", "qift_fused_mnz.hip", "qift_fwht.h", "qift_internal.h", "qift_mma.h")


def _sources_hash() -> str:
    """Digest of the decode kernel's sources: a committed traffic record is used only while it matches."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_02823_amd", "csrc")
    for f in DECODE_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def _environment(torch):
    """GPU, target, ROCm/HIP and torch versions, and the clocks rocm-smi reports (a child process)."""
    props = torch.cuda.get_device_properties(0)
    env = {"gpu": torch.cuda.get_device_name(0), "arch": getattr(props, "gcnArchName", None),
           "hip": torch.version.hip, "torch": torch.__version__, "cus": props.multi_processor_count}
    try:
        import subprocess
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=20)
        env["clocks"] = [ln.strip() for ln in r.stdout.splitlines() if "clk" in ln.lower() and "(" in ln][:8]
    except Exception as e:   # the tool may be missing; the bench line does not depend on it
        env["clocks"] = f"unavailable: {type(e).__name__}"
    return env


def _traffic_record():
    """HBM bytes per launch of the decode kernel from the committed rocprofv3 PMC summary.

    Returns None unless the summary was taken on the current kernel sources.
    """
    path = os.path.join(ROOT, "profiles", "decode_fused_cfg1_m1_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("sources_sha") != _sources_hash():
        return None
    return rec.get("bytes_per_launch")


class DecodeStack:
    """cfg1 layer shapes x 32 distinct layers, M tokens, MNZ."""

    def __init__(self, torch, qift, synth, layers=32, M=1, fused=True):
        self.torch, self.qift, self.synth = torch, qift, synth
        self.layers, self.M, self.fused = layers, M, fused
        c = synth.CONFIGS[1]
        sh = {s.name: s for s in c.linears}
        # (name, N, K, block, activation site); q|k|v and gate|up stacked along N
        self.plan = [("qkv", 3 * sh["q"].N, sh["q"].K, sh["q"].block, 0),
                     ("o", sh["o"].N, sh["o"].K, sh["o"].block, 1),
                     ("gate_up", 2 * sh["gate"].N, sh["gate"].K, sh["gate"].block, 2),
                     ("down", sh["down"].N, sh["down"].K, sh["down"].block, 3)]
        self.workload = ("LLaMA-2-7B-shaped decode layer (q,k,v,o 4096x4096; gate,up 11008x4096; "
                         "down 4096x11008, Hadamard 4096 / 172x64), MNZ W2, M=%d; 32 distinct seeded "
                         "layers per step (q|k|v and gate|up stacked along N)" % M)

    def setup(self):
        torch, qift, synth = self.torch, self.qift, self.synth
        dev = torch.device("cuda")
        c = synth.CONFIGS[1]
        self.weights, self.x, self.acts, self.outs = [], [], [], []
        for layer in range(self.layers):
            ws = []
            for slot, (name, N, K, b, site) in enumerate(self.plan):
                lev = synth.draw_levels_torch(qift.W2_MNZ, N, K, seed=1_000_003 * layer + slot, device=dev)
                sc = torch.from_numpy(synth.draw_scales(qift.W2_MNZ, N, cfg=1, layer=layer, slot=slot)).to(dev)
                ws.append(qift.pack_w2(lev, sc, qift.W2_MNZ))
                del lev
            self.weights.append(ws)
            self.x.append([torch.from_numpy(synth.config_activations(c, layer, site, self.M, K)).to(dev)
                           for (_, _, K, _, site) in self.plan])
        self.acts = [qift.alloc_act(self.M, K, dev) for (_, _, K, _, _) in self.plan]
        self.outs = [torch.empty((self.M, N), dtype=torch.float16, device=dev) for (_, N, _, _, _) in self.plan]
        torch.cuda.synchronize()
        self.packed_bytes = sum(w.nbytes for ws in self.weights for w in ws)
        # algorithmic bytes of one linear launch: packed words + fp16 scales + the activation it
        # reads (fp16 x when the rotation is fused, else int8 act_q + fp32 scale + int32 sum)
        # + fp16 output
        M = self.M
        act_b = (lambda K: 2 * M * K) if self.fused else (lambda K: M * K + 8 * M)
        self.alg_bytes = [N * K // 4 + 2 * N + act_b(K) + 2 * M * N for (_, N, K, _, _) in self.plan]

    def step(self):
        """One token through the stack: per linear, rotate + quantize its input, then the linear."""
        qift = self.qift
        for layer in range(self.layers):
            ws, xs = self.weights[layer], self.x[layer]
            for i, (name, N, K, b, site) in enumerate(self.plan):
                if self.fused:
                    qift.rotate_quant_linear(ws[i], xs[i], b, out=self.outs[i])
                else:
                    act = qift.rotate_quant_act(xs[i], b, out=self.acts[i])
                    qift.w2a4_linear(ws[i], act, out=self.outs[i])

    def linear_launches(self):
        """Only the launches of the decode linear kernel of one step."""
        qift = self.qift
        for layer in range(self.layers):
            for i, (name, N, K, b, site) in enumerate(self.plan):
                if self.fused:
                    qift.rotate_quant_linear(self.weights[layer][i], self.x[layer][i], b, out=self.outs[i])
                else:
                    qift.w2a4_linear(self.weights[layer][i], self.acts[i], out=self.outs[i])

    @property
    def launches_per_step(self):
        return self.layers * len(self.plan)


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
                qift.linear(ws[i], act, out=self.outs[i])


class SweepStack:
    """32 distinct seeded layers of one config at M tokens: cfg2 (LLaMA-3.1-8B, MNZ; q|k|v, o, gate|up,
    down) or cfg3 (LLaMA-3.1-8B MLP, PoT; gate|up, down).  M = 1 runs the fused rotate+linear entry,
    larger M one rotate_quant_act per input and the linear on its codes (the decode kernel per block
    of 16 tokens up to M = 64)."""

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
                    qift.w2a4_linear(ws[i], act, out=self.outs[i])


def stack_sweep(torch, qift, synth, reps=20):
    """Tokens/s and packed GB/s of the cfg2 stack at M in {1, 4, 16} and the cfg3 PoT MLP stack at
    M in {1, 8, 64} (hipGraph replays, inputs resident)."""
    rows = []
    for cfg, Ms in ((2, (1, 4, 16)), (3, (1, 8, 64))):
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
    """Each decode shape's kernel looped over >= min_bytes of distinct weight replicas (M = 1)."""
    c = synth.CONFIGS[1]
    sh = {s.name: s for s in c.linears}
    plan = [("q,k,v", 3 * sh["q"].N, sh["q"].K, sh["q"].block, 0), ("o", sh["o"].N, sh["o"].K, sh["o"].block, 1),
            ("gate,up", 2 * sh["gate"].N, sh["gate"].K, sh["gate"].block, 2),
            ("down", sh["down"].N, sh["down"].K, sh["down"].block, 3)]
    rows = []
    for name, N, K, b, site in plan:
        dev = torch.device("cuda")
        lev = synth.draw_levels_torch(qift.W2_MNZ, N, K, seed=99 + site, device=dev)
        sc = torch.from_numpy(synth.draw_scales(qift.W2_MNZ, N, cfg=1, layer=0, slot=site)).to(dev)
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
                qift.w2a4_linear(w, act, out=y)

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
                qift.w2a4_linear(w, act, out=y)
        t = _time_graph(torch, mnz, reps)
        row["mnz_integer_us"] = round(t / R * 1e6, 2)
        rows.append(row)
        del reps_w, reps_i, base
        torch.cuda.empty_cache()
    return {"workload": "LLaMA-2-7B-shaped decode linears (cfg1), M = 1, activation codes precomputed; "
                        "random 2-bit codes (the kernel's work does not depend on them)", "rows": rows}


FP64_VECTOR_PEAK_TFLOPS = 78.6
POT_FLOPS_PER_WEIGHT = 64 * 5   # per candidate: w / s, compare, s * level, w - s * level, d * d + acc


def weight_quantizer(torch, qift, synth, reps=5):
    """The GPU weight quantizer on one LLaMA-3.1-8B layer (its 7 linears, 218M fp32 weights) per
    format: rotation, per-row scale and levels (the offline step before packing; hipGraph replays,
    weights resident).  MNZ and W4 move 4 B in + 1 B out per weight (HBM roofline); the PoT scale
    search is fp64 arithmetic, priced at 5 flops per candidate and weight against the fp64 vector
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


def cpu_baseline(synth, budget_s=20.0):
    """The oracle as it stands, on one cfg1 layer at M=1 (4 act quantizations + 7 linears)."""
    import numpy as np
    from oracle import levels as olev, linear as olin, pack as opack, quant
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    c = synth.CONFIGS[1]
    sites = {}
    prepared = []
    for s in c.linears:
        L = synth.draw_levels(olev.FMT_W2_MNZ, s.N, s.K, cfg=1, layer=0, slot=synth.LINEAR_ID[s.name])
        sw = synth.draw_scales(olev.FMT_W2_MNZ, s.N, cfg=1, layer=0, slot=synth.LINEAR_ID[s.name])
        prepared.append((s, opack.pack_qw2(L, olev.FMT_W2_MNZ), sw))
        site = synth.SITE_OF[s.name]
        sites.setdefault(site, (synth.config_activations(c, 0, site, 1, s.K), s.block))
    packed = sum(P.nbytes for _, P, _ in prepared)

    def one_layer():
        qa = {site: quant.act_quant(x, b) for site, (x, b) in sites.items()}
        for s, P, sw in prepared:
            q, sx, _, _ = qa[synth.SITE_OF[s.name]]
            olin.linear(P, sw, olev.FMT_W2_MNZ, s.K, q, sx)

    one_layer()                         # warm the oracle's cached Hadamard matrices
    t0 = time.perf_counter()
    n = 0
    while True:
        one_layer()
        n += 1
        if time.perf_counter() - t0 > budget_s / 2 or n >= 2:
            break
    dt = (time.perf_counter() - t0) / n

    def parts(with_pack):
        """Seconds of one layer's activation quantizations and linears, measured apart, and of packing
        the levels of one 4096 x 4096 linear (its own rate, not scaled to the layer)."""
        a0 = time.perf_counter()
        qa = {site: quant.act_quant(x, b) for site, (x, b) in sites.items()}
        a1 = time.perf_counter()
        for s, P, sw in prepared:
            q, sx, _, _ = qa[synth.SITE_OF[s.name]]
            olin.linear(P, sw, olev.FMT_W2_MNZ, s.K, q, sx)
        a2 = time.perf_counter()
        r = {"act_quant_s": round(a1 - a0, 3), "linears_s": round(a2 - a1, 3),
             "layer_GBs": round(packed / (a2 - a0) / 1e9, 4)}
        if with_pack:
            p0 = time.perf_counter()
            P = opack.pack_qw2(pack_levels, olev.FMT_W2_MNZ)
            p1 = time.perf_counter()
            r["pack_4096x4096_s"] = round(p1 - p0, 3)
            r["pack_GBs_of_packed"] = round(P.nbytes / (p1 - p0) / 1e9, 4)
        return r

    sq = next(s for s in c.linears if s.name == "q")
    pack_levels = synth.draw_levels(olev.FMT_W2_MNZ, sq.N, sq.K, cfg=1, layer=0, slot=synth.LINEAR_ID["q"])
    detail = {"all_threads": parts(True)}
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(1):
            detail["one_thread"] = parts(False)
    except Exception as e:  # pragma: no cover
        detail["one_thread"] = f"unavailable: {type(e).__name__}"
    try:
        with open("/proc/cpuinfo") as f:
            detail["cpu_model"] = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:  # pragma: no cover
        detail["cpu_model"] = None
    return {"value": round(packed / dt / 1e9, 4), "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one cfg1 layer (7 linears, 4 activation quantizations) at M=1, {n} timed pass(es) "
                      f"of {dt:.2f} s after one warm-up; {packed} packed bytes per pass; host has "
                      f"{os.cpu_count()} logical CPUs",
            "detail": detail}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--prefill-steps", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="launch the decode step eagerly")
    ap.add_argument("--unfused", action="store_true",
                    help="decode step as separate rotate_quant_act + w2a4_linear launches")
    ap.add_argument("--no-per-shape", action="store_true",
                    help="skip the per-shape replica loops and the read probe")
    ap.add_argument("--no-wquant", action="store_true", help="skip the weight quantizer timing")
    ap.add_argument("--no-kv4", action="store_true", help="skip the KV4 attention timing")
    ap.add_argument("--no-lut", action="store_true", help="skip the level-table linear timing")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the cfg2 (M 1/4/16) and cfg3 PoT (M 1/8/64) stack sweep")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run 1 GiB device copies (HBM byte-counter calibration under rocprofv3)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the quantized linear shards by output rows with no "
              "exchange, so the job throughput is the per-GPU figure; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_02823_amd import qift, synth
    qift.lib()
    torch.cuda.set_device(0)

    # ---------------------------------------------------------------- decode (headline)
    _stage("decode step")
    dec = DecodeStack(torch, qift, synth, layers=args.layers, M=1, fused=not args.unfused)
    dec.setup()
    dec.step()                                   # eager warm-up
    torch.cuda.synchronize()
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            dec.step()
        torch.cuda.current_stream().wait_stream(s)
        with torch.cuda.graph(graph):
            dec.step()
    run = graph.replay if graph is not None else dec.step
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

    # per-launch duration of the decode kernel: HIP events around back-to-back replays of a graph
    # holding just this step's linear launches (same stream, shapes and weights); inside a graph
    # the launches run without gaps, so this is the kernel's own average duration
    lin_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(lin_graph):
        dec.linear_launches()
    lin_graph.replay()
    torch.cuda.synchronize()
    la, lb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    la.record()
    for _ in range(args.steps):
        lin_graph.replay()
    lb.record()
    torch.cuda.synchronize()
    avg_dur = la.elapsed_time(lb) * 1e-3 / (args.steps * dec.launches_per_step)
    del lin_graph
    bytes_per_launch = sum(dec.alg_bytes) / len(dec.alg_bytes)
    achieved = bytes_per_launch / avg_dur / 1e9
    traffic = _traffic_record()
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": DECODE_KERNEL if args.unfused else DECODE_KERNEL_FUSED,
                "avg_launch_us": round(avg_dur * 1e6, 3),
                "alg_bytes_per_launch": int(bytes_per_launch)}
    stack_kernel_sum_ms = avg_dur * dec.launches_per_step * 1e3

    out = {"metric": METRIC, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "i8xi2->i32", "data": "synthetic",
           "config": {"workload": dec.workload, "tokens_per_step": dec.M, "layers": dec.layers,
                      "packed_bytes_per_step": dec.packed_bytes, "launch": "hipGraph" if graph else "eager",
                      "rotation": "separate rotate_quant_act" if args.unfused else "fused into each linear"},
           "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
           "tokens_per_s": round(dec.M / (ms * 1e-3), 1),
           "host_wall_s": round(wall, 3),
           "stack_kernel_sum_ms": round(stack_kernel_sum_ms, 4),
           "step_ms_distribution": step_dist,
           "roofline": roofline,
           "env": _environment(torch)}
    del graph
    dec = None
    torch.cuda.empty_cache()

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
        pre.step()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.prefill_steps):
            pre.step()
        b.record()
        torch.cuda.synchronize()
        pms = a.elapsed_time(b) / args.prefill_steps
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
                    dt = _time_graph(torch, lambda: qift.linear(w, pre.acts[i], out=pre.outs[i], workspace=ws), 10)
                    per_shape.append({"linear": name, "format": fname, "path": path, "N": N, "K": K,
                                      "us": round(dt * 1e6, 2), "int8_tops": round(ops / dt / 1e12, 2),
                                      "pct_int8_peak": round(100 * ops / dt / 1e12 / INT8_PEAK_TOPS, 2)})
        out["prefill"] = {"workload": "LLaMA-3.1-8B-shaped prefill, M=2048, layers 0-15 W4 / 16-31 W2 MNZ, "
                                      "4 rotate_quant_act + 4 linears per layer (q|k|v and gate|up stacked "
                                      "along N)",
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
