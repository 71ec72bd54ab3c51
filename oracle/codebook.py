"""Non-uniform codebooks for KVQuant-style quantization: 1-D Lloyd k-means.

The paper only says KVQuant stores values with b bits (Section 2.1).  The
non-uniform 2^b-entry codebook is read here as the minimum-squared-error
(Lloyd) quantizer of the normalised non-outlier values of a separate
calibration draw:
  * samples are sorted ascending; centroid i starts at sample
    floor((2i + 1) * N / (2K)) (the (i + 1/2)/K quantile), K = 2^b;
  * each Lloyd iteration assigns every sample to its nearest centroid (ties to
    the lower index) and moves each centroid to the mean of its samples; a
    centroid with no samples keeps its value;
  * iteration stops when no assignment changes, or after max_iter iterations;
  * the codebook is stored like every other value of the cache, in fp16: the
    final centroids are rounded (once, to nearest even) to fp16 and sorted
    ascending (returned as float32 holding fp16 values).

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import numpy as np


def lloyd_centroids(samples, bits, max_iter=100, chunk=1 << 18):
    """Lloyd centroids in float64 (unrounded), in centroid-index order."""
    x = np.sort(np.asarray(samples, np.float64).ravel())
    n = x.size
    kk = 1 << int(bits)
    if n == 0:
        raise ValueError("no calibration samples")
    idx = np.minimum(n - 1, ((2 * np.arange(kk) + 1) * n) // (2 * kk))
    c = x[idx].copy()
    assign = None
    for _ in range(max_iter):
        new = np.empty(n, np.int64)
        for a in range(0, n, chunk):
            xs = x[a:a + chunk]
            new[a:a + chunk] = np.argmin(np.abs(xs[:, None] - c[None, :]), axis=1)
        if assign is not None and np.array_equal(new, assign):
            break
        assign = new
        sums = np.bincount(assign, weights=x, minlength=kk)
        cnts = np.bincount(assign, minlength=kk)
        c = np.where(cnts > 0, sums / np.maximum(cnts, 1), c)
    return c


def lloyd_codebook(samples, bits, max_iter=100, chunk=1 << 18):
    """The stored codebook: Lloyd centroids rounded to fp16, ascending, as float32."""
    c = lloyd_centroids(samples, bits, max_iter, chunk)
    return np.sort(c.astype(np.float16).astype(np.float32))
