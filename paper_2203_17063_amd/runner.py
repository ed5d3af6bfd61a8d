"""Device-side drivers over the C ABI: upload host arrays with torch (device
memory and streams only) and call libecc.  No arithmetic of the method runs
here."""
from __future__ import annotations

import numpy as np
import torch

from . import capi as E


def _dev(a, dtype=None, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device)


def ptr_array(tensors, device="cuda"):
    """Device array of the data pointers of `tensors` (for d_send, d_fresh, d_slots)."""
    return torch.tensor([t.data_ptr() for t in tensors], dtype=torch.int64, device=device)


def current_stream():
    return torch.cuda.current_stream().cuda_stream


class Plan:
    """Owns an ecc_plan_t."""

    def __init__(self, P, counts, displs, S, stream=None):
        self.P = int(P)
        self.handle = E.ecc_plan_create(self.P, counts, displs, int(S),
                                        current_stream() if stream is None else stream)

    def reset(self):
        E.ecc_plan_reset(self.handle)

    def stats(self):
        return E.ecc_plan_stats(self.handle, self.P)

    def close(self):
        if self.handle:
            E.ecc_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Iterative:
    """An iterative problem resident in HBM: CSR matrix, block layout, arrival
    table, right-hand side, and the iterate buffers."""

    def __init__(self, n, row_ptr, col, val, counts, S, mask, kind, b=None, alpha=0.0,
                 beta=0.0, x0=None, device="cuda", range_bytes=0, tile_rows=0, schedule=0,
                 compact=0):
        self.n = int(n)
        self.kind = kind
        self.alpha, self.beta = float(alpha), float(beta)
        self.counts = np.asarray(counts, dtype=np.int64)
        self.P = len(self.counts)
        displs = np.zeros(self.P, dtype=np.int64)
        displs[1:] = np.cumsum(self.counts[:-1])
        self.d_row_ptr = _dev(row_ptr, device=device)
        self.d_col = _dev(col, device=device)
        self.d_val = _dev(val, device=device)
        self.nnz = int(len(col))
        self.d_mask = _dev(np.asarray(mask, dtype=np.uint8), device=device)
        self.T = int(mask.shape[0])
        self.d_b = _dev(b, device=device) if b is not None else None
        self.x0 = np.zeros(self.n) if x0 is None else np.asarray(x0, dtype=np.float64)
        # x0 stays resident: each solve restarts from it with a device copy
        self.d_x0 = _dev(self.x0, device=device)
        self.d_x = torch.empty(self.n, dtype=torch.float64, device=device)
        self.d_x_tmp = torch.empty_like(self.d_x)
        self.d_x_hat = torch.empty_like(self.d_x)
        self.d_rho = torch.zeros(max(self.T, 1), dtype=torch.float64, device=device)
        self.plan = Plan(self.P, self.counts, displs, S)
        self.csr = E.make_csr(self.n, self.n, self.nnz, self.d_row_ptr, self.d_col, self.d_val)
        ekind = E.ECC_KIND_JACOBI if kind == "jacobi" else E.ECC_KIND_POWER
        self.mat = E.ecc_matrix_create_ex(self.plan.handle, self.csr, ekind, range_bytes,
                                          tile_rows, schedule, compact)
        self.d_partials = torch.empty(E.ecc_partials_size(self.mat), dtype=torch.float64,
                                      device=device)

    def load_x0(self):
        if self.n:
            E.ecc_stream_copy(self.d_x, self.d_x0, self.n, current_stream())

    def solve(self, T=None, tol=0.0, histories=False):
        """Reset the plan, load x0 and run T iterations through ecc_solve.
        Returns the number of iterations run."""
        T = self.T if T is None else T
        self.plan.reset()
        self.load_x0()
        eff = age = None
        if histories:
            eff = torch.empty((T, self.P), dtype=torch.uint8, device=self.d_x.device)
            age = torch.empty((T, self.P), dtype=torch.int32, device=self.d_x.device)
        self.eff_hist, self.age_hist = eff, age
        return E.ecc_solve(self.plan.handle, self.mat, self.d_b, self.alpha, self.beta,
                           self.d_x, self.d_x_tmp, self.d_x_hat, self.d_mask, T, tol,
                           self.d_rho, eff, age)

    def step(self, t, x_own, x_next, eff_out=None, age_out=None):
        """One iteration through the separate calls: assemble, sweep, norm.
        Returns the norm (synchronising)."""
        E.ecc_allgatherv_assemble_packed(self.plan.handle, x_own, self.d_x_hat,
                                         self.d_mask[t].data_ptr(), eff_out, age_out)
        if self.kind == "jacobi":
            E.ecc_iterate_jacobi(self.plan.handle, self.mat, self.d_b, x_own, self.d_x_hat,
                                 x_next, self.d_partials)
            norm = E.ECC_NORM_L2
        else:
            E.ecc_iterate_spmv(self.plan.handle, self.mat, self.alpha, self.beta, x_own,
                               self.d_x_hat, x_next, self.d_partials)
            norm = E.ECC_NORM_L1
        return E.ecc_residual(self.plan.handle, self.d_partials, self.d_partials.numel(), norm)

    def close(self):
        if getattr(self, "mat", None):
            E.ecc_matrix_destroy(self.mat)
            self.mat = None
        if getattr(self, "plan", None):
            self.plan.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class MatrixFactorization:
    """Data-parallel matrix factorisation over the partial allreduce: ratings,
    model, per-worker gradient and slot buffers resident in HBM; every
    iteration is enqueued through ecc_mf_iterate."""

    def __init__(self, prob, device="cuda"):
        self.prob = prob
        P, m = prob.P, prob.m
        self.d_users = _dev(prob.users, device=device)
        self.d_items = _dev(prob.items, device=device)
        self.d_ratings = _dev(prob.ratings, device=device)
        self.d_W0 = _dev(prob.W0, device=device)
        self.d_W = self.d_W0.clone()
        self.grads = [torch.empty(m, dtype=torch.float64, device=device) for _ in range(P)]
        self.slots = [torch.zeros(m, dtype=torch.float64, device=device) for _ in range(P)]
        self.d_grads = ptr_array(self.grads, device)
        self.d_slots = ptr_array(self.slots, device)
        self.d_G = torch.empty(m, dtype=torch.float64, device=device)
        self.d_mask = _dev(np.asarray(prob.mask, dtype=np.uint8), device=device)
        self.d_batch = _dev(np.asarray(prob.batch, dtype=np.int32), device=device)
        self.d_rmse = torch.zeros(max(prob.T, 1), dtype=torch.float64, device=device)
        self.d_err = torch.zeros(max(prob.T, 1) + 1, dtype=torch.float64, device=device)
        self.d_eff = torch.zeros((max(prob.T, 1), P), dtype=torch.uint8, device=device)
        self.plan = Plan(P, None, None, prob.S)
        self.handle = E.ecc_mf_create(prob.n_users, prob.n_items, prob.rank, P, prob.K, prob.N,
                                      self.d_users, self.d_items, self.d_ratings)

    def reset(self):
        self.plan.reset()
        self.d_W.copy_(self.d_W0)

    def iterate(self, t, record=True, error=False):
        """Iteration t; with error, also the full training error at the model
        on entry into d_err[t]."""
        if error:
            E.ecc_mf_error(self.handle, self.d_W, self.d_err[t].data_ptr(), current_stream())
        E.ecc_mf_iterate(self.handle, self.plan.handle, self.prob.eta, self.prob.lam, self.d_W,
                         self.d_grads, self.d_slots, self.d_G, self.d_mask[t].data_ptr(),
                         self.d_batch[t].data_ptr(), self.d_rmse[t].data_ptr(),
                         self.d_eff[t] if record else None)

    def run(self, T=None, record=True, errors=False):
        """T iterations from W0; with errors, the full training error before
        every iteration and after the last (d_err[0 .. T])."""
        T = self.prob.T if T is None else T
        self.reset()
        for t in range(T):
            self.iterate(t, record, errors)
        if errors:
            E.ecc_mf_error(self.handle, self.d_W, self.d_err[T].data_ptr(), current_stream())

    def close(self):
        if getattr(self, "handle", None):
            E.ecc_mf_destroy(self.handle)
            self.handle = None
        if getattr(self, "plan", None):
            self.plan.close()
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
