"""Calibrates the peak offsets used by workloads.synth (run once; prints the constants).

Targets, from the workload descriptions: the small workload (T = 32768, V = 32768) has a mean
sampled-token training confidence of about 0.8; the long-response workload (V = 151936) has
about 80% of its tokens with sampled training probability above 0.95. The training probability of a sampled id is read off torch.softmax of
the pilot rows (a library routine; this script is not part of the loss path).

    python -m workloads.calibrate
"""

import torch

from workloads import synth


def sampled_p(cfg: int, peak: float, frac: float, rows: int = 256, seed: int = 123):
    old = (synth.PEAK_1, synth.PEAK_3, synth.PEAK_3_FRACTION)
    synth.PEAK_1, synth.PEAK_3, synth.PEAK_3_FRACTION = peak, peak, frac
    try:
        b = synth.make_batch(cfg, device="cpu", seed=seed, rows=rows, rows_per_step=64)
    finally:
        synth.PEAK_1, synth.PEAK_3, synth.PEAK_3_FRACTION = old
    p = torch.softmax(b.logits.float(), dim=1).gather(1, b.ids[:, None])[:, 0]
    return p


def main():
    lo, hi = 0.0, 12.0
    for _ in range(18):
        mid = 0.5 * (lo + hi)
        if sampled_p(1, mid, 0.0).mean() < 0.80:
            lo = mid
        else:
            hi = mid
    print(f"PEAK_1 = {0.5 * (lo + hi):.2f}   (mean sampled p = {sampled_p(1, 0.5 * (lo + hi), 0).mean():.3f})")
    peak3 = 9.0
    lo, hi = 0.5, 1.0
    for _ in range(14):
        mid = 0.5 * (lo + hi)
        if (sampled_p(3, peak3, mid) > 0.95).float().mean() < 0.80:
            lo = mid
        else:
            hi = mid
    f = 0.5 * (lo + hi)
    p = sampled_p(3, peak3, f)
    print(f"PEAK_3 = {peak3}  PEAK_3_FRACTION = {f:.2f}   (share p > 0.95 = {(p > 0.95).float().mean():.3f},"
          f" peaked-row p median = {p[p > 0.5].median():.5f})")


if __name__ == "__main__":
    main()
