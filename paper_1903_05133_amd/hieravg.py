"""Python handle over the C ABI (marshalling only).  Device memory for outputs
and the stream come from PyTorch; the replicas, dataset and every kernel live
in the HIP library."""

import ctypes

import numpy as np

from . import native


class HierAvg:
    """One Hier-AVG job: P learners of one model as rows of one replica array.

    Construct either from a named workload (``model`` = 0..3, see
    ``include/hieravg.h``) or from a ``native.Config``.
    """

    def __init__(self, P=None, S=None, K1=None, K2=None, model=None, lr=None, B=None, seed=0, config=None):
        L = native.lib()
        if config is not None:
            self._cfg = config
            h = L.hieravg_create_config(ctypes.byref(config))
        else:
            self._cfg = None
            h = L.hieravg_create(P, S, K1, K2, model, lr, B, seed)
        if not h:
            raise native.HierAvgError(L.hieravg_last_error().decode())
        self._h = h
        self.P = P if config is None else config.P
        self.K1 = K1 if config is None else config.K1
        self.K2 = K2 if config is None else config.K2
        self.B = B if config is None else config.B
        self.T = self.K1 * self.K2 if config is None or config.k_global == 0 else config.k_global
        self.D = int(L.hieravg_dim(h))

    # -------------------------------------------------------------- lifecycle
    def close(self):
        if getattr(self, "_h", None):
            native.lib().hieravg_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -------------------------------------------------------------- the method
    def round(self):
        native.check(native.lib().hieravg_round(self._h))

    def sync(self):
        native.check(native.lib().hieravg_sync(self._h))

    @property
    def steps(self):
        return int(native.lib().hieravg_step_count(self._h))

    # -------------------------------------------------------------- state
    def params_into(self, ptr, n_floats):
        native.check(native.lib().hieravg_params(self._h, ctypes.c_void_p(ptr), n_floats))

    def params(self, device=None):
        """All replicas as [P, D] float32: a numpy array, or a torch tensor on
        ``device`` when one is given."""
        if device is None:
            out = np.empty((self.P, self.D), dtype=np.float32)
            self.params_into(out.ctypes.data, out.size)
            return out
        import torch
        out = torch.empty((self.P, self.D), dtype=torch.float32, device=device)
        self.params_into(out.data_ptr(), out.numel())
        return out

    def set_params(self, arr):
        if hasattr(arr, "data_ptr"):
            native.check(native.lib().hieravg_set_params(self._h, ctypes.c_void_p(arr.data_ptr()), arr.numel()))
        else:
            a = np.ascontiguousarray(arr, dtype=np.float32)
            native.check(native.lib().hieravg_set_params(self._h, ctypes.c_void_p(a.ctypes.data), a.size))

    def finite(self):
        """True when every replica holds finite values (divergence check)."""
        rc = native.lib().hieravg_check_finite(self._h)
        if rc == native.ENONFINITE:
            return False
        native.check(rc)
        return True

    def set_step_count(self, t):
        """Global step counter: the next round draws its minibatches for steps t, t+1, ..."""
        native.check(native.lib().hieravg_set_step_count(self._h, t))

    def state(self):
        """Checkpoint at a round boundary: replicas, momentum buffers (None
        without momentum), global step count."""
        try:
            mom = self.momentum()
        except native.HierAvgError:
            mom = None
        return {"params": self.params(), "momentum": mom, "steps": self.steps}

    def load_state(self, st):
        """Resume from state(): the rounds that follow are those of the
        uninterrupted run."""
        self.set_params(st["params"])
        if st.get("momentum") is not None:
            self.set_momentum(st["momentum"])
        self.set_step_count(int(st["steps"]))

    def save(self, path):
        """Write state() to an .npz file (plain arrays, no pickled objects)."""
        st = self.state()
        arrays = {"params": st["params"], "steps": np.array(st["steps"], dtype=np.int64)}
        if st["momentum"] is not None:
            arrays["momentum"] = st["momentum"]
        np.savez(path, **arrays)

    def load(self, path):
        with np.load(path, allow_pickle=False) as z:
            self.load_state({"params": z["params"], "steps": int(z["steps"]),
                             "momentum": z["momentum"] if "momentum" in z.files else None})

    def momentum(self):
        """Momentum buffers of all learners as [P, D] float32 (numpy)."""
        out = np.empty((self.P, self.D), dtype=np.float32)
        native.check(native.lib().hieravg_momentum(self._h, ctypes.c_void_p(out.ctypes.data), out.size))
        return out

    def set_momentum(self, arr):
        a = np.ascontiguousarray(arr, dtype=np.float32)
        native.check(native.lib().hieravg_set_momentum(self._h, ctypes.c_void_p(a.ctypes.data), a.size))

    def set_batch(self, B):
        """Minibatch size of the rounds that follow (at most the B at create)."""
        native.check(native.lib().hieravg_set_batch(self._h, B))
        self.B = B

    def set_lr(self, lr):
        """Step size of the rounds that follow."""
        native.check(native.lib().hieravg_set_lr(self._h, lr))

    def evaluate(self, replica=0, split=1, n_rows=4096):
        """(mean cross-entropy, correct count) of replica `replica` on
        `n_rows` training (split 0) or held-out (split 1) rows."""
        loss = ctypes.c_double()
        correct = ctypes.c_int64()
        native.check(native.lib().hieravg_evaluate(self._h, replica, split, n_rows, ctypes.byref(loss),
                                                   ctypes.byref(correct)))
        return loss.value, correct.value

    def last_indices(self):
        """Indices of the last round: [K2, K1, P, B], or [T, P, B] when the
        round length T is not K1 * K2."""
        shape = (self.K2, self.K1, self.P, self.B) if self.T == self.K1 * self.K2 else (self.T, self.P, self.B)
        out = np.empty(shape, dtype=np.int32)
        native.check(native.lib().hieravg_last_indices(self._h, ctypes.c_void_p(out.ctypes.data), out.size))
        return out

    def set_stream(self, stream):
        """Enqueue on a torch stream (or a raw hipStream_t int; None = own)."""
        handle = None if stream is None else (stream if isinstance(stream, int) else stream.cuda_stream)
        native.check(native.lib().hieravg_set_stream(self._h, ctypes.c_void_p(handle)))

    # -------------------------------------------------------------- timing
    def profile(self, enable=True):
        native.check(native.lib().hieravg_profile(self._h, 1 if enable else 0))

    def time_kernel(self, name, reps=100):
        """Mean ms of one launch of kernel class `name` over `reps` back-to-back
        launches (changes the replicas: measurement only)."""
        L = native.lib()
        names = [L.hieravg_kernel_class_name(i).decode() for i in range(L.hieravg_kernel_classes())]
        ms = ctypes.c_double()
        native.check(L.hieravg_time_kernel(self._h, names.index(name), reps, ctypes.byref(ms)))
        return ms.value

    def profile_read(self):
        """{kernel class name: (launches, total ms)} of the recorded launches."""
        L = native.lib()
        n = L.hieravg_kernel_classes()
        launches = (ctypes.c_int64 * n)()
        ms = (ctypes.c_double * n)()
        native.check(L.hieravg_profile_read(self._h, launches, ms, n))
        return {L.hieravg_kernel_class_name(i).decode(): (int(launches[i]), float(ms[i]))
                for i in range(n) if launches[i]}


def config(kind, P, S, K1, K2, B=1, in_dim=0, hidden=0, classes=0, n_samples=0, noise_std=1.0, lr=0.05,
           momentum=0.0, init_std=0.01, grad_std=0.01, seed=0, update_mode=0, k_global=0, weight_decay=0.0,
           avg_momentum=False):
    return native.Config(P=P, S=S, K1=K1, K2=K2, B=B, kind=kind, in_dim=in_dim, hidden=hidden, classes=classes,
                         n_samples=n_samples, noise_std=noise_std, lr=lr, momentum=momentum, init_std=init_std,
                         grad_std=grad_std, seed=seed, update_mode=update_mode, k_global=k_global,
                         weight_decay=weight_decay, avg_momentum=1 if avg_momentum else 0)
