"""A CPU engine for the recovery-protocol tests: one rank's flat shard held
in host memory and committed by the oracle (test infrastructure; the product
engine keeps the shard on the GPU and commits it through libpactshard).  The
gradient of update t is drawn from (seed, t) at the shard's global indices,
as on the GPU."""
import numpy as np

import oracle
import workloads as wl


class OracleEngine:
    def __init__(self, numel, global_offset, seed, hyper=None):
        self.n, self.goff, self.seed = int(numel), int(global_offset), int(seed)
        self.hyper = oracle.Hyper(**(hyper or {}))
        self.p = wl.draw(self.n, self.goff, self.seed, wl.ARRAY_PARAM, 0, wl.NORMAL(0.02))
        self.g = np.zeros(self.n, np.float32)
        self.m = np.zeros(self.n, np.float32)
        self.v = np.zeros(self.n, np.float32)
        self.b = np.zeros(self.n, np.uint16)

    def produce_grad(self, step):
        wl.fill_host(self.g, self.goff, self.seed, wl.ARRAY_GRAD, step, wl.NORMAL(1e-3))

    def commit(self, step, torn=False):
        k = self.n // 2 if torn else self.n
        d = oracle.commit_and_digest(self.p[:k], self.g[:k], self.m[:k], self.v[:k], self.b[:k], self.hyper, step,
                                     self.goff)
        oracle.zero_grad(self.g)
        return d

    def outstanding(self):
        return oracle.count_outstanding(self.g)

    def digest(self):
        return oracle.state_digest(self.p, self.m, self.v, self.goff)

    def synchronize(self):
        pass

    def save(self, path):
        np.savez(path, p=self.p, m=self.m, v=self.v)

    def load(self, path):
        with np.load(path, allow_pickle=False) as z:
            self.p, self.m, self.v = (np.ascontiguousarray(z[k]) for k in ("p", "m", "v"))
        self.g[:] = 0.0
