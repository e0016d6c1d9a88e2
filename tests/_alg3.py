"""Alg. 3 (SGD with SDP4Bit) on a least-squares problem with W = P*Q
simulated data-parallel workers, driving the compression path end to end.

Per step:
  1. every worker computes the gradient of its row block at the model
     weights w~ (host, float32 numpy -- identical for every backend);
  2. gradient compression U_g = the two-level path run as a reduce-scatter:
     worker (a, b) quantizes its gradient (Hadamard + 8-bit); "GPU" (a, b)
     reduces chunk b of the 8-bit messages of node a and re-quantizes to
     4 bits; "GPU" (a', b) reduces chunk a' of the 4-bit messages of every
     node (inverse Hadamard, out_scale 1/W) into its shard [b*M + a'*m, ...);
  3. main weights w <- w - eta * g;
  4. weight communication: qWD (w~ <- w~ + C(w - w~), the model-weight update of Alg. 3), or
     qW (w~ <- C(w), direct quantization), or none (w~ = w).

Two backends compute steps 2 and 4: the CPU oracle and the HIP library.
"""
import numpy as np

import oracle


class Problem:
    def __init__(self, d=2048, rows=8192, P=4, Q=2, group=128, block=256, seed=0, noise=0.1):
        r = np.random.default_rng(seed)
        self.d, self.P, self.Q, self.W = d, P, Q, P * Q
        self.group, self.block = group, block
        self.A = r.standard_normal((rows, d)).astype(np.float32)
        self.w_star = r.standard_normal(d).astype(np.float32)
        self.b = (self.A @ self.w_star + noise * r.standard_normal(rows)).astype(np.float32)
        self.rows_per = rows // self.W
        self.M = d // P
        self.m = self.M // Q

    def loss(self, w):
        res = self.A.astype(np.float64) @ w.astype(np.float64) - self.b
        return 0.5 * float(res @ res) / self.A.shape[0]

    def worker_grads(self, w):
        out = []
        for k in range(self.W):
            Ak = self.A[k * self.rows_per:(k + 1) * self.rows_per]
            bk = self.b[k * self.rows_per:(k + 1) * self.rows_per]
            out.append((Ak.T @ (Ak @ w - bk) / np.float32(self.rows_per)).astype(np.float32))
        return out


class OracleBackend:
    def __init__(self, pb: Problem):
        self.pb = pb

    def reduce_scatter(self, grads):
        pb = self.pb
        P, Q, M, m, g, nb = pb.P, pb.Q, pb.M, pb.m, pb.group, pb.block
        k1 = [oracle.grad_quant(x, 8, nb, g)[:2] for x in grads]          # worker k = a*P + b
        level2 = {}
        for a in range(Q):
            for b in range(P):
                cs = [k1[a * P + bb][0][b * M:(b + 1) * M] for bb in range(P)]
                ss = [k1[a * P + bb][1][b * M // g:(b + 1) * M // g] for bb in range(P)]
                r = oracle.dequant_reduce(cs, ss, M, 8, g, 4, want_f32=False)
                level2[a, b] = (r["codes"], r["scales"])
        out = np.empty(pb.d, np.float32)
        for a2 in range(Q):
            for b in range(P):
                cs = [level2[a, b][0][a2 * m // 2:(a2 + 1) * m // 2] for a in range(Q)]
                ss = [level2[a, b][1][a2 * m // g:(a2 + 1) * m // g] for a in range(Q)]
                f = oracle.dequant_reduce(cs, ss, m, 4, g, 0, nb, 1.0 / pb.W)["f32"]
                out[b * M + a2 * m:b * M + (a2 + 1) * m] = f
        return out

    def qwd(self, w, wt, group):
        c, s, mn, _ = oracle.qwd_encode(w, wt, group)
        return oracle.qwd_decode(c, s, mn, wt, group)

    def qw(self, w, group):
        zero = np.zeros_like(w)
        c, s, mn, _ = oracle.qwd_encode(w, zero, group)
        return oracle.qwd_decode(c, s, mn, zero, group)


class GpuBackend:
    """The same steps through the HIP library (device buffers via torch)."""

    def __init__(self, pb: Problem):
        import torch
        from paper_2410_15526_amd import sdp4
        self.torch, self.sdp4, self.pb = torch, sdp4, pb
        e = lambda k, dt: torch.empty(k, dtype=dt, device="cuda")
        W, d, M, g = pb.W, pb.d, pb.M, pb.group
        self.x = e(W * d, torch.float32)
        self.c8 = e(W * d, torch.uint8)
        self.s8 = e(W * d // g, torch.float32)
        self.c4 = e(W * M // 2, torch.uint8)                 # (a, b) -> slot a*P + b
        self.s4 = e(W * M // g, torch.float32)
        self.out = e(d, torch.float32)
        self.wq = e(d, torch.float32)
        self.wt = e(d, torch.float32)
        self.qc = e(d // 2, torch.uint8)
        self.qs = e(d, torch.float32)
        self.qm = e(d, torch.float32)

    def reduce_scatter(self, grads):
        t, L, pb = self.torch, self.sdp4, self.pb
        P, Q, M, m, g, nb, d = pb.P, pb.Q, pb.M, pb.m, pb.group, pb.block, pb.d
        self.x.copy_(t.from_numpy(np.concatenate(grads)))
        for k in range(pb.W):
            L.sdp4_grad_quant(self.x[k * d:(k + 1) * d], 8, nb, g, self.c8[k * d:(k + 1) * d],
                              self.s8[k * d // g:(k + 1) * d // g])
        for a in range(Q):
            for b in range(P):
                cs = [self.c8[(a * P + bb) * d + b * M:(a * P + bb) * d + (b + 1) * M] for bb in range(P)]
                ss = [self.s8[((a * P + bb) * d + b * M) // g:((a * P + bb) * d + (b + 1) * M) // g]
                      for bb in range(P)]
                slot = a * P + b
                L.sdp4_dequant_reduce(cs, ss, M, 8, g, 4, 0, 1.0, self.c4[slot * M // 2:(slot + 1) * M // 2],
                                      self.s4[slot * M // g:(slot + 1) * M // g])
        for a2 in range(Q):
            for b in range(P):
                cs = [self.c4[(a * P + b) * M // 2 + a2 * m // 2:(a * P + b) * M // 2 + (a2 + 1) * m // 2]
                      for a in range(Q)]
                ss = [self.s4[((a * P + b) * M + a2 * m) // g:((a * P + b) * M + (a2 + 1) * m) // g]
                      for a in range(Q)]
                L.sdp4_dequant_reduce(cs, ss, m, 4, g, 0, nb, 1.0 / pb.W, None, None,
                                      self.out[b * M + a2 * m:b * M + (a2 + 1) * m])
        t.cuda.synchronize()
        return self.out.cpu().numpy().copy()

    def qwd(self, w, wt, group):
        t, L = self.torch, self.sdp4
        d = w.size
        self.wq.copy_(t.from_numpy(w))
        self.wt.copy_(t.from_numpy(wt))
        qs, qm = self.qs[:d // group], self.qm[:d // group]
        L.sdp4_qwd_encode(self.wq, self.wt, group, self.qc, qs, qm)
        L.sdp4_qwd_decode(self.qc, qs, qm, group, self.wt)
        t.cuda.synchronize()
        return self.wt.cpu().numpy().copy()

    def qw(self, w, group):
        return self.qwd(w, np.zeros_like(w), group)


def train(pb: Problem, backend, mode: str, steps: int, eta: float, weight_group: int = 128,
          compress_grads: bool = True, record=None):
    """mode: 'full' (w~ = w), 'qwd' (Alg. 3), 'qw' (w~ = C(w)).  Returns the loss history."""
    w = np.zeros(pb.d, np.float32)
    wt = w.copy()
    hist = [pb.loss(wt)]
    for _ in range(steps):
        grads = pb.worker_grads(wt)
        g = backend.reduce_scatter(grads) if compress_grads else \
            (np.sum(np.stack(grads).astype(np.float64), axis=0) / pb.W).astype(np.float32)
        w = (w - np.float32(eta) * g).astype(np.float32)
        if mode == "full":
            wt = w.copy()
        elif mode == "qwd":
            wt = backend.qwd(w, wt, weight_group)
        else:
            wt = backend.qw(w, weight_group)
        hist.append(pb.loss(wt))
        if record is not None:
            record.append(wt.copy())
    return hist
