"""Helpers of the GPU parity tests: run the HIP library through the C ABI on
seeded inputs, and compare with the oracle under the normalised tolerance.

Tolerance.  A float32 result x computed on the GPU is accepted when
    |x_gpu - x_ref| <= rtol * S_abs(x)
where S_abs(x) is the sum of the absolute values of every term that forms x
(forward: sum |w|; SGD weight: |w_old| + lr * A with A = sum |contributions|;
Adagrad state: s_old + A^2; Adagrad weight: |w_old| + lr * A / (sqrt(s_new)
+ eps)).  rtol = 1e-5 for float32 storage, 1e-2 for bfloat16 storage.
Since S_abs >= |x_ref| this is the plain relative error whenever no
cancellation happens; it is needed because float32 sums taken in atomic
order over tens of thousands of N(0,1) terms carry an absolute error of the
order u * sum |terms|, which plain relative error on a cancelled sum cannot
bound.
"""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss

RTOL = {"f32": 1e-5, "bf16": 1e-2}


SIGN_FLAG = {None: 0, "pm1": pss.PSS_SIGN_PM1, "sparse": pss.PSS_SIGN_SPARSE}


class Layer:
    """One workload's device state: shared array (+ Adagrad state) and params.

    Options: sign in (None, "pm1", "sparse"), mean pooling, int32 indices and
    offsets (idx32), bfloat16 pooled rows (rows_bf16)."""

    def __init__(self, wl, B=None, batch=0, M=None, flags=pss.PSS_BWD_AUTO, s0=0.0, w=None,
                 sign=None, mean=False, idx32=False, rows_bf16=False):
        self.wl = wl if M is None else wl.scaled(M=M)
        wl = self.wl
        self.B = wl.B if B is None else B
        self.x = synth.make_inputs(wl, B=self.B, batch=batch)
        self.a, self.b = o.hash_params_from_seed(wl.hash_seed)
        self.dev = torch.device("cuda", 0)
        self.w_host = synth.make_weights(wl) if w is None else w
        if wl.weight_dtype == "bf16":
            self.shared = torch.from_numpy(self.w_host.view(np.int16)).to(self.dev).view(torch.bfloat16)
        else:
            self.shared = torch.from_numpy(self.w_host).to(self.dev)
        self.s_host = None
        self.state = None
        if wl.optimizer == "adagrad":
            self.s_host = np.full(wl.M, s0, dtype=np.float32)
            self.state = torch.from_numpy(self.s_host).to(self.dev)
        itype = torch.int32 if idx32 else torch.int64
        self.indices = torch.from_numpy(self.x.indices).to(self.dev).to(itype)
        self.offsets = torch.from_numpy(self.x.offsets).to(self.dev).to(itype)
        self.sign_mode, self.mean, self.rows_bf16 = sign, mean, rows_bf16
        flags |= SIGN_FLAG[sign] | (pss.PSS_POOL_MEAN if mean else 0)
        flags |= (pss.PSS_INDEX_I32 if idx32 else 0) | (pss.PSS_ROWS_BF16 if rows_bf16 else 0)
        self.hp = pss.make_hash_params(wl.hash_seed, num_tables=wl.T, batch=self.B,
                                       num_indices=self.x.N,
                                       weight_dtype=pss.PSS_BF16 if wl.weight_dtype == "bf16" else pss.PSS_F32,
                                       eps=wl.eps, flags=flags)
        assert (self.hp.a, self.hp.b) == (self.a, self.b)
        self.sign = None if sign is None else (sign,) + o.sign_params_from_seed(wl.hash_seed)

    def forward(self):
        """Pooled rows as float32 (bfloat16 rows widened exactly)."""
        wl = self.wl
        dt = torch.bfloat16 if self.rows_bf16 else torch.float32
        out = torch.empty((self.B, wl.T * wl.d), dtype=dt, device=self.dev)
        pss.pss_forward(self.shared, wl.M, wl.Z, wl.d, self.hp, self.indices, self.offsets, out)
        torch.cuda.synchronize()
        return out.float().cpu().numpy()

    def grad_values(self, grad_host):
        """The gradient values the library reads: bfloat16 rows are rounded
        (nearest even) from the float32 draw; both sides use these."""
        if not self.rows_bf16:
            return grad_host
        return torch.from_numpy(grad_host).to(torch.bfloat16).float().numpy()

    def backward(self, grad_host, lr=None):
        wl = self.wl
        g = torch.from_numpy(grad_host)
        if self.rows_bf16:
            g = g.to(torch.bfloat16)  # on the host, as grad_values
        g = g.to(self.dev)
        pss.pss_backward_update(self.shared, self.state, wl.M, wl.Z, wl.d, self.hp, self.indices,
                                self.offsets, g, wl.lr if lr is None else lr)
        torch.cuda.synchronize()

    def weights(self):
        if self.wl.weight_dtype == "bf16":
            return self.shared.view(torch.int16).cpu().numpy().view(np.uint16)
        return self.shared.cpu().numpy()

    def debug_signs(self):
        wl = self.wl
        out = torch.empty((self.x.N, wl.C), dtype=torch.int8, device=self.dev)
        pss.pss_debug_signs(wl.M, wl.Z, wl.d, self.hp, self.indices, self.offsets, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    def debug_bases(self):
        wl = self.wl
        out = torch.empty((self.x.N, wl.C), dtype=torch.int32, device=self.dev)
        pss.pss_debug_addresses(wl.M, wl.Z, wl.d, self.hp, self.indices, self.offsets, out)
        torch.cuda.synchronize()
        return out.cpu().numpy().view(np.uint32)

    # oracle side ---------------------------------------------------------
    def ref_forward(self):
        wl = self.wl
        return o.forward64(self.w_host, wl.M, wl.Z, wl.d, wl.T, self.B, self.a, self.b,
                           self.x.indices, self.x.offsets, wl.weight_dtype, sign=self.sign,
                           mean=self.mean)

    def ref_backward(self, grad_host, lr=None):
        wl = self.wl
        return o.backward_update(self.w_host, self.s_host, wl.M, wl.Z, wl.d, wl.T, self.B, self.a,
                                 self.b, self.x.indices, self.x.offsets, self.grad_values(grad_host),
                                 wl.lr if lr is None else lr, wl.eps, wl.weight_dtype,
                                 sign=self.sign, mean=self.mean)


def check_forward(got, ref64, s_abs, rtol, rows_bf16=False):
    """rows_bf16: the float32 result was rounded once more to bfloat16, which
    adds at most half a bfloat16 ulp (2^-9 relative) of the value."""
    err = np.abs(got.astype(np.float64) - ref64)
    bound = rtol * s_abs + 1e-30
    if rows_bf16:
        bound = bound + 2.0**-8 * (np.abs(ref64) + rtol * s_abs)
    bad = err > bound
    assert not bad.any(), (f"{bad.sum()} of {bad.size} outputs out of tolerance; worst "
                           f"normalised error {(err / np.maximum(s_abs, 1e-300)).max():.3e}")
    return float((err / np.maximum(s_abs, 1e-300)).max())


def check_update(layer, w_gpu, s_gpu, w_ref, s_ref, G, A, lr):
    """Element-wise check of an SGD/Adagrad update against the oracle."""
    wl = layer.wl
    rtol = RTOL[wl.weight_dtype]
    w_old = o.widen(layer.w_host, wl.weight_dtype)
    wg = o.widen(w_gpu, wl.weight_dtype)
    wr = o.widen(w_ref, wl.weight_dtype)
    exempt = np.zeros(wg.shape, dtype=bool)
    if s_gpu is None:
        bound_w = np.abs(w_old) + lr * A
    else:
        s_old = layer.s_host.astype(np.float64)
        s_new = s_ref.astype(np.float64)
        bound_s = s_old + A * A
        err_s = np.abs(s_gpu.astype(np.float64) - s_new)
        bad_s = err_s > rtol * bound_s + 1e-30
        assert not bad_s.any(), f"{bad_s.sum()} Adagrad states out of tolerance"
        bound_w = np.abs(w_old) + lr * A / (np.sqrt(s_new) + wl.eps)
        # first step from s = 0 is discontinuous at G = 0: the sign of a
        # cancelled sum decides a move of about lr; such elements are exempt
        exempt = (s_old == 0) & (np.abs(G) <= rtol * A)
    err_w = np.abs(wg - wr)
    bad_w = (err_w > rtol * bound_w + 1e-30) & ~exempt
    assert not bad_w.any(), (f"{bad_w.sum()} weights out of tolerance; worst normalised "
                             f"{(err_w / np.maximum(bound_w, 1e-300))[~exempt].max():.3e}")
    # elements no lookup touched keep their exact bits
    untouched = A == 0
    if wl.weight_dtype == "bf16":
        assert np.array_equal(w_gpu[untouched], layer.w_host[untouched])
    else:
        assert np.array_equal(w_gpu[untouched].view(np.uint32), layer.w_host[untouched].view(np.uint32))
    return int(exempt.sum())
