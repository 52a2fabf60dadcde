"""Adversarial shifted-score sets for the P-gen unit (test helper, no method
arithmetic): scores placed on every code threshold and every scale-exponent
boundary of Alg. 1 (within +-2 fp32 ulps), masked keys and blocks, denormal
and tiny scores, and block maxima below the E8M0 range."""
import math

import numpy as np

LN2 = math.log(2.0)


def adversarial_scores(rng, rows, cols, tau, h):
    """Shifted scores with exact code thresholds, k-boundaries, masked keys,
    denormals and very negative block maxima."""
    x = -rng.exponential(2.5, size=(rows, cols)).astype(np.float32)
    nblk = (cols + 31) // 32
    for r in range(rows):
        kind = r % 6
        for b in range(nblk):
            t0 = b * 32
            n = min(32, cols - t0)
            if kind == 0:       # block max 0 -> k = -3; neighbours of every threshold
                x[r, t0] = 0.0
                for i in range(1, n):
                    c = (i - 1) % 7
                    xt = np.float32(tau + c / h - 3 * LN2 + math.log(6.0))
                    step = (i - 1) // 7 - 2   # -2..+2 ulps
                    v = xt
                    for _ in range(abs(step)):
                        v = np.nextafter(v, np.float32(np.inf if step > 0 else -np.inf))
                    x[r, t0 + i] = min(v, np.float32(0.0))
            elif kind == 1:     # block maxima at and around k boundaries
                j = -3 - (b % 20)
                Mb = np.float32(j * LN2 - math.log(2 / 9))
                d = (r // 6 + b) % 5 - 2
                for _ in range(abs(d)):
                    Mb = np.nextafter(Mb, np.float32(np.inf if d > 0 else -np.inf))
                x[r, t0] = min(Mb, np.float32(0.0))
            elif kind == 2:     # masked keys
                mask = rng.random(n) < 0.5
                x[r, t0:t0 + n][mask] = -np.inf
                if b % 3 == 0:
                    x[r, t0:t0 + n] = -np.inf
            elif kind == 3:     # denormals and tiny values
                x[r, t0:t0 + n] = -rng.uniform(0, 1e-37, n).astype(np.float32)
                x[r, t0 + 1] = -np.float32(1e-42)
            elif kind == 4:     # block maximum below the E8M0 range
                x[r, t0:t0 + n] -= np.float32(80 + (b % 10))
    return x
