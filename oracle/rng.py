"""Counter-based randomness of the oracle: minibatch draw and synthetic inputs.

TEST INFRASTRUCTURE ONLY (see the package docstring).

In Algorithm 1 (Sec. 3.1) every learner draws a fresh random minibatch of B
samples at each local step; Sec. 2 makes the samples i.i.d. across learners
and iterations.  The paper
names no generator, so the reading used here is a counter-based one that any
implementation can reproduce bit for bit:

  * H(key, c) = mix64(key + (c + 1) * 0x9E3779B97F4A7C15 mod 2^64), the output
    function of SplitMix64 (Steele, Lea & Flood, "Fast splittable
    pseudorandom number generators", OOPSLA 2014) evaluated at counter c.
  * sample s of learner j at global SGD step t:
        idx = H(key_index, (t << 32) | (j << 16) | s) mod N      (unsigned)
    i.e. i.i.d. draws with replacement; the bit fields do not depend on P or B.
  * stream keys: key_tag = H(seed, TAG) for the fixed 64-bit tags below.

Synthetic inputs (stand-ins for the paper's image data) use an exact normal
surrogate so that every value is a float32 number reproducible on any
hardware: z = (sum of the twelve 16-bit fields of H(key, 3e), H(key, 3e+1),
H(key, 3e+2)) - 393210) / 65536, an Irwin-Hall(12) variate with mean 0 and
variance 1 - 2^-32.

All arithmetic on uint64 arrays wraps modulo 2^64, as the definition requires.
"""

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
MIX_M1 = 0xBF58476D1CE4E5B9
MIX_M2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

# Stream tags: the ASCII bytes of the names, big-endian.
TAG_INDEX = int.from_bytes(b"hv.index", "big")
TAG_LABEL = int.from_bytes(b"hv.label", "big")
TAG_MEAN = int.from_bytes(b"hv.cmean", "big")
TAG_NOISE = int.from_bytes(b"hv.noise", "big")
TAG_INIT = int.from_bytes(b"hv.winit", "big")
TAG_GRAD = int.from_bytes(b"hv.grads", "big")
# held-out rows: same class means, their own labels and noise
TAG_TEST_LABEL = int.from_bytes(b"hv.tlabl", "big")
TAG_TEST_NOISE = int.from_bytes(b"hv.tnois", "big")

IRWIN_HALL_OFFSET = 393210  # 12 * (2^16 - 1) / 2
IRWIN_HALL_SCALE = 65536.0


# ---------------------------------------------------------------- scalar form
def mix64_scalar(z: int) -> int:
    """SplitMix64 output mixing function on a Python int (mod 2^64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX_M1) & MASK64
    z = ((z ^ (z >> 27)) * MIX_M2) & MASK64
    return z ^ (z >> 31)


def h_scalar(key: int, counter: int) -> int:
    """H(key, c) on Python ints."""
    return mix64_scalar((key + ((counter + 1) * GOLDEN)) & MASK64)


def splitmix64_sequence(state: int, n: int) -> list:
    """The SplitMix64 generator stepped n times from `state` (published form:
    state += golden; output mix64(state)).  Equal to H(state, 0..n-1)."""
    out = []
    for _ in range(n):
        state = (state + GOLDEN) & MASK64
        out.append(mix64_scalar(state))
    return out


def stream_key(seed: int, tag: int) -> int:
    return h_scalar(seed & MASK64, tag)


# ---------------------------------------------------------------- array form
def _u64(x):
    return np.asarray(x, dtype=np.uint64)


def mix64(z):
    z = _u64(z)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX_M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX_M2)
        return z ^ (z >> np.uint64(31))


def h(key: int, counter):
    """Vectorised H(key, c) for a uint64 array of counters."""
    c = _u64(counter)
    with np.errstate(over="ignore"):
        return mix64(np.uint64(key) + (c + np.uint64(1)) * np.uint64(GOLDEN))


def draw_indices(seed: int, learner: int, step: int, B: int, N: int):
    """Indices of the B samples learner `learner` uses at global step `step`."""
    key = stream_key(seed, TAG_INDEX)
    s = np.arange(B, dtype=np.uint64)
    ctr = (np.uint64(step) << np.uint64(32)) | (np.uint64(learner) << np.uint64(16)) | s
    return (h(key, ctr) % np.uint64(N)).astype(np.int64)


def normal_surrogate(key: int, e):
    """Exact Irwin-Hall(12) normal surrogate at element counters `e` (float64
    array whose values are exactly representable in float32)."""
    e = _u64(e)
    acc = np.zeros(e.shape, dtype=np.int64)
    with np.errstate(over="ignore"):
        for r in range(3):
            v = h(key, e * np.uint64(3) + np.uint64(r))
            for f in range(4):
                acc += ((v >> np.uint64(16 * f)) & np.uint64(0xFFFF)).astype(np.int64)
    return (acc - IRWIN_HALL_OFFSET).astype(np.float64) / IRWIN_HALL_SCALE


def labels(seed: int, rows, C: int, split: int = 0):
    key = stream_key(seed, TAG_LABEL if split == 0 else TAG_TEST_LABEL)
    return (h(key, _u64(rows)) % np.uint64(C)).astype(np.int64)


def class_means(seed: int, classes, IN: int):
    """mu[c, d] for the requested classes (float64 holding float32 values)."""
    key = stream_key(seed, TAG_MEAN)
    classes = np.asarray(classes, dtype=np.uint64).reshape(-1, 1)
    d = np.arange(IN, dtype=np.uint64).reshape(1, -1)
    return normal_surrogate(key, classes * np.uint64(IN) + d)


def data_rows(seed: int, rows, IN: int, C: int, sigma: float, split: int = 0):
    """Rows X[i, :] and labels y[i] of the synthetic dataset (split 0) or of
    the held-out set (split 1: the same class means, its own label and noise
    streams), regenerated on demand (never materialised):
    X = fp32(mu[y] + sigma * z)."""
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    y = labels(seed, rows, C, split)
    uniq, inv = np.unique(y, return_inverse=True)
    mu = class_means(seed, uniq, IN)[inv]
    key = stream_key(seed, TAG_NOISE if split == 0 else TAG_TEST_NOISE)
    d = np.arange(IN, dtype=np.uint64).reshape(1, -1)
    z = normal_surrogate(key, rows.astype(np.uint64).reshape(-1, 1) * np.uint64(IN) + d)
    sig = float(np.float32(sigma))
    x = (mu + sig * z).astype(np.float32).astype(np.float64)
    return x, y


def init_uniform(seed: int, layer: int, rows: int, cols: int):
    """Initial weight matrix [rows, cols] of layer `layer`: (2u - 1) * s with
    u = (H >> 40) * 2^-24 and s = fp32(1 / sqrt(cols)) (fan-in scaling)."""
    key = stream_key(seed, TAG_INIT)
    s = float(np.float32(1.0 / np.sqrt(float(cols))))
    w = np.empty(rows * cols, dtype=np.float64)
    step = 1 << 20  # elements per piece (the values do not depend on it)
    for a in range(0, rows * cols, step):
        e = (np.uint64(layer) << np.uint64(48)) + np.arange(a, min(a + step, rows * cols), dtype=np.uint64)
        u = (h(key, e) >> np.uint64(40)).astype(np.float64) * 2.0 ** -24
        w[a:a + len(e)] = ((2.0 * u - 1.0) * s).astype(np.float32)
    return w.reshape(rows, cols)


def init_vector(seed: int, D: int, std: float, cols=None):
    """Initial replica of the averaging-only workload: fp32(std * z); only the
    coordinates `cols` when given (coordinates never interact)."""
    key = stream_key(seed, TAG_INIT)
    d = np.arange(D, dtype=np.uint64) if cols is None else np.asarray(cols, dtype=np.uint64)
    z = normal_surrogate(key, d)
    return (float(np.float32(std)) * z).astype(np.float32).astype(np.float64)


def given_gradients(seed: int, k: int, learner: int, D: int, std: float, cols=None):
    """Gradient handed to learner `learner` at step-in-round k in the
    averaging-only workload: fp32(std * z) at counters (k*2^16 + j)*D + d
    (only the coordinates `cols` when given)."""
    key = stream_key(seed, TAG_GRAD)
    base = (np.uint64(k) * np.uint64(65536) + np.uint64(learner)) * np.uint64(D)
    d = np.arange(D, dtype=np.uint64) if cols is None else np.asarray(cols, dtype=np.uint64)
    z = normal_surrogate(key, base + d)
    return (float(np.float32(std)) * z).astype(np.float32).astype(np.float64)
