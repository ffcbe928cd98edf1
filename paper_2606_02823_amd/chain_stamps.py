"""Phase breakdown of the persistent decode chain from the diagnostic build's wall-clock stamps.

    python -m paper_2606_02823_amd.build --stamps
    python -m paper_2606_02823_amd.chain_stamps [layers]

Runs the LLaMA-3.1-8B decode step (q|k|v 6144x4096, o 4096x4096, gate|up 28672x4096, down 4096x14336
with Hadamard blocks of 2048; MNZ weights, M = 1, real data dependencies) for `layers` layers (default
4, at most 16: the stamps cover the first 64 links) through libqift_stamps.so, reads the stamps of the
last call and prints, per linear shape, the median over workgroups and over the layers after the
first of each phase of a link (microseconds):

  visible   the median producer of the previous link is done (its stores complete) -> this
            workgroup's input is in
  spread    the last producer's done time minus the median producer's
  rotation  input in -> the activation group's rotation is done
  max       rotation done -> the token's max is known
  quantize  max known -> the codes are in LDS
  barrier   codes in LDS -> weight wave 4 passed the codes barrier
  mfma      that barrier -> wave 4's MFMAs are done
  tail      MFMAs done -> the last weight wave of the workgroup is done (its stores complete)
  link      median producer to median producer

The stamps are global stores of their own, so a stamped step is slightly slower than the product's.
"""
from __future__ import annotations

import ctypes
import os
import sys

import numpy as np

PLAN = [("q|k|v", 6144, 4096, 4096), ("o", 4096, 4096, 4096), ("gate|up", 28672, 4096, 4096),
        ("down", 4096, 14336, 2048)]
N_WG, N_LINK, N_MARK = 256, 64, 32


def main(layers: int = 4) -> None:
    import torch
    from . import qift, synth
    qift.LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libqift_stamps.so")
    L = qift.lib()
    L.qift_chain_stamps_read.restype = ctypes.c_int
    L.qift_chain_stamps_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t]
    dev = torch.device("cuda")
    layers = max(2, min(layers, N_LINK // len(PLAN)))
    links, keep = [], []
    for l in range(layers):
        base = len(links)
        for s, (_, N, K, b) in enumerate(PLAN):
            lev = synth.draw_levels_torch(qift.W2_MNZ, N, K, seed=1000 * l + s, device=dev)
            sc = torch.full((N,), 1.0 / (1.7 * np.sqrt(K)), dtype=torch.float16, device=dev)
            pk = qift.pack_w2(lev, sc, qift.W2_MNZ)
            del lev
            keep.append(pk)
            src = (base - 1 if l else -1) if s == 0 else base + s - 1
            links.append(qift.ChainLink(pk, b, src, 0))
    chain = qift.Chain(links, 1)
    x = torch.from_numpy(synth.config_activations(synth.CONFIGS[2], 0, 0, 1, 4096)).to(dev)
    for _ in range(3):
        chain.run(x)
    torch.cuda.synchronize()
    err = qift.device_error()
    buf = np.zeros(N_WG * N_LINK * N_MARK, dtype=np.uint64)
    st = L.qift_chain_stamps_read(buf.ctypes.data, buf.nbytes)
    if st != 0:
        raise RuntimeError(f"qift_chain_stamps_read: {st}")
    n = len(links)
    d = buf.reshape(N_WG, N_LINK, N_MARK)[:, :n, :].astype(np.float64)
    t0 = np.nanmin(np.where(d[:, 0, 1] > 0, d[:, 0, 1], np.nan))
    d = np.where(d > 0, (d - t0) / 100.0, np.nan)   # 100 MHz ticks -> microseconds
    stores = np.nanmax(d[:, :, 16:24], axis=2)       # per workgroup and link: its last weight wave done
    med = lambda a: float(np.nanmedian(a))
    print(f"LLaMA-3.1-8B decode step, MNZ, M = 1, {layers} layers ({n} links), stamps of the last call; "
          f"device error bits {err}")
    print()
    print("| link | visible | spread | rotation | max | quantize | barrier | mfma | tail | link |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    total = 0.0
    for s, (name, N, K, _) in enumerate(PLAN):
        rows = []
        for i in range(len(PLAN) + s, n, len(PLAN)):
            prev_med, prev_last = med(stores[:, i - 1]), float(np.nanmax(stores[:, i - 1]))
            rows.append([med(d[:, i, 1]) - prev_med, prev_last - prev_med,
                         med(d[:, i, 2] - d[:, i, 1]), med(d[:, i, 3] - d[:, i, 2]), med(d[:, i, 4] - d[:, i, 3]),
                         med(d[:, i, 5] - d[:, i, 4]), med(d[:, i, 6] - d[:, i, 5]),
                         med(stores[:, i] - d[:, i, 6]), med(stores[:, i]) - prev_med])
        r = np.median(np.array(rows), axis=0)
        total += r[-1]
        label = name.replace("|", "\\|")   # a table cell
        print(f"| {label} {N}x{K} | " + " | ".join(f"{v:.2f}" for v in r) + " |")
    print()
    print(f"per layer: {total:.2f} us")


if __name__ == "__main__":
    main(int(sys.argv[1]) if len(sys.argv) > 1 else 4)
