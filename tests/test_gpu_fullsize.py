"""Full-size parity: every workload at its real size, through the same entry
points and launch configuration that bench.py times (default backward
variant; the step as the bench runs it, with PSS_PREPARE_BACKWARD on the
forward, for the one-hot and multi-hot workloads), checked on sampled
outputs the oracle evaluates one by one: pooled rows of sampled bags
(forward_at) and updated weights at sampled elements of the shared array
(gradient_at), half of them elements that the batch reads.

Alg. 1's sparse branch at full size as well: the SPARSE backward variant on
every workload (sampled elements, as above), and the exported sparse
gradient (pss_gradient_sparse) on the workloads whose arrays fit the export:
its location count equals the number of distinct elements the batch reads
(the union of the oracle's chunk windows), its locations ascend strictly,
every sampled element the batch reads is listed with the oracle's value, and
no sampled element it does not read is listed.

The run sums by address (opt-in, whole-row chunks) at full size on the
row-hash workload, with and without the prepared grouping: bit-identical."""
import numpy as np
import pytest
import torch

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss

pytestmark = pytest.mark.gpu

FULL = ["c2", "c3", "c4", "c5"]
RTOL = {"f32": 1e-5, "bf16": 1e-2}


class Full:
    def __init__(self, key, flags=0):
        print(f"full-size {key}: preparing inputs", flush=True)
        self.wl = wl = synth.get(key)
        self.x = synth.make_inputs(wl)
        self.w = synth.make_weights(wl)
        self.dev = torch.device("cuda", 0)
        if wl.weight_dtype == "bf16":
            self.shared = torch.from_numpy(self.w.view(np.int16)).to(self.dev).view(torch.bfloat16)
        else:
            self.shared = torch.from_numpy(self.w).to(self.dev)
        self.state = torch.zeros(wl.M, device=self.dev) if wl.optimizer == "adagrad" else None
        self.idx = torch.from_numpy(self.x.indices).to(self.dev)
        self.off = torch.from_numpy(self.x.offsets).to(self.dev)
        self.hp = pss.make_hash_params(
            wl.hash_seed, num_tables=wl.T, batch=wl.B, num_indices=self.x.N, eps=wl.eps,
            weight_dtype=pss.PSS_BF16 if wl.weight_dtype == "bf16" else pss.PSS_F32, flags=flags)
        self.a, self.b = self.hp.a, self.hp.b


@pytest.mark.parametrize("key", FULL)
def test_fullsize_forward_sampled_bags(key):
    F = Full(key)
    wl = F.wl
    out = torch.empty((wl.B, wl.T * wl.d), dtype=torch.float32, device=F.dev)
    print(f"full-size {key}: forward over {F.x.N} lookups", flush=True)
    pss.pss_forward(F.shared, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, out)
    torch.cuda.synchronize()
    _check_forward(F, out)


def _check_forward(F, out):
    wl = F.wl
    rng = np.random.default_rng(100)
    nb = wl.T * wl.B
    bags = np.unique(np.concatenate([rng.choice(nb, 300, replace=False),
                                     [0, nb - 1, wl.B - 1, wl.B, nb - 64, nb - 65]]))
    t, b = bags // wl.B, bags % wl.B
    got = out.view(wl.B, wl.T, wl.d)[torch.from_numpy(b).to(F.dev), torch.from_numpy(t).to(F.dev)]
    got = got.cpu().numpy().astype(np.float64)
    ref, s_abs = o.forward_at(F.w, wl.M, wl.Z, wl.d, wl.T, wl.B, F.a, F.b, F.x.indices,
                              F.x.offsets, bags, wl.weight_dtype)
    bad = np.abs(got - ref) > 1e-5 * s_abs + 1e-30
    assert not bad.any(), f"{bad.sum()} of {bad.size} sampled outputs out of tolerance"


def _sample_elements(F, rng, n_read=1500, n_any=500):
    wl = F.wl
    e = rng.choice(F.x.N, size=min(n_read, F.x.N), replace=False)
    _, t_all, _ = o.item_bags(wl.T, wl.B, F.x.offsets)
    addr = o.addresses_from_bases(wl.M, wl.Z, o.bases_for(wl.M, wl.Z, wl.d, wl.T, F.a, F.b,
                                                          F.x.indices[e], t_all[e]))
    read = addr[np.arange(e.shape[0]), rng.integers(0, wl.d, e.shape[0])]
    anyw = rng.integers(0, wl.M, n_any)
    return np.unique(np.concatenate([read, anyw, [0, wl.M - 1]]))


def _grad(F):
    """N(0, 1) output gradient drawn on the device (seeded), and its host
    copy for the oracle."""
    wl = F.wl
    gen = torch.Generator(device=F.dev).manual_seed(wl.data_seed)
    g = torch.randn((wl.B, wl.T * wl.d), device=F.dev, generator=gen)
    return g, g.cpu().numpy()


@pytest.mark.parametrize("key", FULL)
def test_fullsize_backward_sampled_elements(key):
    F = Full(key)
    wl = F.wl
    g, grad = _grad(F)
    print(f"full-size {key}: backward over {F.x.N} lookups", flush=True)
    pss.pss_backward_update(F.shared, F.state, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, wl.lr)
    torch.cuda.synchronize()
    del g
    _check_backward(F, grad)


@pytest.mark.parametrize("key", ["c2", "c3"])
def test_fullsize_prepared_step(key):
    """The bench's step: forward with PSS_PREPARE_BACKWARD, then the backward
    reusing the grouping (one-hot: the streamed forward kernel writes its
    keygen stage and the backward finishes it; multi-hot: the grouping runs
    on the library's stream beside the forward kernel)."""
    F = Full(key, flags=pss.PSS_PREPARE_BACKWARD)
    wl = F.wl
    g, grad = _grad(F)
    out = torch.empty((wl.B, wl.T * wl.d), dtype=torch.float32, device=F.dev)
    torch.cuda.synchronize()
    print(f"full-size {key}: prepared step over {F.x.N} lookups", flush=True)
    pss.pss_forward(F.shared, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, out)
    pss.pss_backward_update(F.shared, F.state, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, wl.lr)
    torch.cuda.synchronize()
    del g
    _check_forward(F, out)
    _check_backward(F, grad)


def _check_backward(F, grad):
    wl = F.wl
    where = _sample_elements(F, np.random.default_rng(200))
    wh = torch.from_numpy(where).to(F.dev)
    if wl.weight_dtype == "bf16":
        w_gpu = F.shared.view(torch.int16)[wh].cpu().numpy().view(np.uint16)
    else:
        w_gpu = F.shared[wh].cpu().numpy()
    print(f"full-size {wl.name}: oracle at {where.shape[0]} elements", flush=True)
    G, A, cnt = o.gradient_at(wl.M, wl.Z, wl.d, wl.T, wl.B, F.a, F.b, F.x.indices, F.x.offsets,
                              grad, where)
    assert (cnt > 0).sum() >= where.shape[0] // 2  # the read elements were sampled
    rtol = RTOL[wl.weight_dtype]
    w_old = F.w[where]
    w_old64 = o.widen(w_old, wl.weight_dtype)
    if F.state is None:
        w_ref = o.sgd_update(w_old, G, wl.lr, wl.weight_dtype)
        bound = np.abs(w_old64) + wl.lr * A
        exempt = np.zeros(where.shape[0], dtype=bool)
    else:
        s_gpu = F.state[wh].cpu().numpy().astype(np.float64)
        w_ref, s_ref = o.adagrad_update(w_old, np.zeros(where.shape[0], np.float32), G, wl.lr,
                                        wl.eps, wl.weight_dtype)
        assert np.all(np.abs(s_gpu - s_ref.astype(np.float64)) <= rtol * A * A + 1e-30)
        bound = np.abs(w_old64) + wl.lr * A / (np.sqrt(s_ref.astype(np.float64)) + wl.eps)
        exempt = np.abs(G) <= rtol * A  # first step from s = 0: sign of a cancelled sum
    err = np.abs(o.widen(w_gpu, wl.weight_dtype) - o.widen(w_ref, wl.weight_dtype))
    bad = (err > rtol * bound + 1e-30) & ~exempt
    assert not bad.any(), f"{bad.sum()} of {where.shape[0]} sampled weights out of tolerance"
    untouched = cnt == 0
    if wl.weight_dtype == "bf16":
        assert np.array_equal(w_gpu[untouched], w_old[untouched])
    else:
        assert np.array_equal(w_gpu[untouched].view(np.uint32), w_old[untouched].view(np.uint32))


@pytest.mark.parametrize("key", FULL)
def test_fullsize_sparse_backward_sampled_elements(key):
    F = Full(key, flags=pss.PSS_BWD_SPARSE)
    wl = F.wl
    g, grad = _grad(F)
    print(f"full-size {key}: SPARSE backward over {F.x.N} lookups", flush=True)
    pss.pss_backward_update(F.shared, F.state, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, wl.lr)
    torch.cuda.synchronize()
    del g
    _check_backward(F, grad)


def _distinct_elements(F):
    """Elements read by the batch: the union of the windows [h, h + Z) mod M
    of the oracle's distinct chunk bases, counted with a difference array."""
    wl = F.wl
    bases = np.unique(o.chunk_bases(wl.M, wl.Z, wl.d, wl.T, wl.B, F.a, F.b, F.x.indices,
                                    F.x.offsets).ravel()).astype(np.int64)
    diff = np.zeros(wl.M + 1, dtype=np.int64)
    end = bases + wl.Z
    np.add.at(diff, bases, 1)
    np.add.at(diff, np.minimum(end, wl.M), -1)
    wrap = end > wl.M  # windows running past the end continue at 0
    np.add.at(diff, np.zeros(int(wrap.sum()), dtype=np.int64), 1)
    np.add.at(diff, end[wrap] - wl.M, -1)
    return int((np.cumsum(diff[:-1]) > 0).sum())


@pytest.mark.parametrize("key", ["c2", "c3", "c5"])
def test_fullsize_gradient_sparse(key):
    F = Full(key)
    wl = F.wl
    g, grad = _grad(F)
    cap = min(wl.M, F.x.N * wl.d)
    loc = torch.empty(cap, dtype=torch.int32, device=F.dev)
    val = torch.empty(cap, dtype=torch.float32, device=F.dev)
    nu = torch.zeros(1, dtype=torch.int64, device=F.dev)
    print(f"full-size {key}: sparse gradient over {F.x.N} lookups", flush=True)
    pss.pss_gradient_sparse(wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, loc, val, nu)
    torch.cuda.synchronize()
    del g
    U = int(nu.item())
    assert U == _distinct_elements(F)
    locs = loc[:U].cpu().numpy().view(np.uint32).astype(np.int64)
    vals = val[:U].cpu().numpy().astype(np.float64)
    assert np.all(np.diff(locs) > 0) and locs[0] >= 0 and locs[-1] < wl.M
    where = _sample_elements(F, np.random.default_rng(300))
    G, A, cnt = o.gradient_at(wl.M, wl.Z, wl.d, wl.T, wl.B, F.a, F.b, F.x.indices, F.x.offsets,
                              grad, where)
    pos = np.searchsorted(locs, where)
    listed = (pos < U) & (locs[np.minimum(pos, U - 1)] == where)
    assert np.array_equal(listed, cnt > 0)
    got = vals[pos[listed]]
    err = np.abs(got - G[listed])
    assert np.all(err <= 1e-5 * A[listed] + 1e-30), f"{(err > 1e-5 * A[listed]).sum()} values off"


def test_fullsize_runs_by_address():
    """Run sums by address on the row-hash workload at full size (its chunks
    are whole rows, Z = 128): the prepared step, sampled elements as above,
    and the same update repeated from the same state bit-identical."""
    flags = pss.PSS_BWD_SORTED | pss.PSS_DEPOSIT_BY_ADDRESS | pss.PSS_PREPARE_BACKWARD
    F = Full("c5", flags=flags)
    wl = F.wl
    g, grad = _grad(F)
    out = torch.empty((wl.B, wl.T * wl.d), dtype=torch.float32, device=F.dev)
    w0, s0 = F.shared.clone(), F.state.clone()
    print(f"full-size c5: run sums by address over {F.x.N} lookups", flush=True)
    pss.pss_forward(F.shared, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, out)
    pss.pss_backward_update(F.shared, F.state, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, wl.lr)
    torch.cuda.synchronize()
    w1, s1 = F.shared.clone(), F.state.clone()
    # again from the same state, without the prepared grouping
    F.shared.copy_(w0)
    F.state.copy_(s0)
    F.hp.flags = pss.PSS_BWD_SORTED | pss.PSS_DEPOSIT_BY_ADDRESS
    pss.pss_backward_update(F.shared, F.state, wl.M, wl.Z, wl.d, F.hp, F.idx, F.off, g, wl.lr)
    torch.cuda.synchronize()
    assert torch.equal(F.shared.view(torch.int16), w1.view(torch.int16))
    assert torch.equal(F.state.view(torch.int32), s1.view(torch.int32))
    del g, w0, s0, w1, s1, out
    _check_backward(F, grad)
