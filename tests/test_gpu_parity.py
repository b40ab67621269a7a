"""GPU parity: the HIP library (through the C ABI) against the CPU oracle.

Sizes are small enough for the oracle to finish in seconds but span many
64-bag tiles with a ragged last tile; the workloads at full size are checked
on sampled outputs in test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu

# (workload, batch, M override) - M kept at full size except where noted
CASES = [("c1", None, None), ("c2", 700, None), ("c3", 50, None), ("c4", 300, 50_000_000),
         ("c5", 900, None)]


VARIANTS = {"atomic": pss.PSS_BWD_ATOMIC, "sorted": pss.PSS_BWD_SORTED,
            "sparse": pss.PSS_BWD_SPARSE}


def _id(c):
    return f"{c[0]}-B{c[1]}"


@pytest.mark.parametrize("case", CASES, ids=_id)
def test_addresses_bit_exact(case):
    key, B, M = case
    L = Layer(synth.get(key), B=B, M=M)
    got = L.debug_bases()
    want = o.chunk_bases(L.wl.M, L.wl.Z, L.wl.d, L.wl.T, L.B, L.a, L.b, L.x.indices, L.x.offsets)
    assert np.array_equal(got.astype(np.uint64), want)


@pytest.mark.parametrize("M", [4096, 2_500_000, 16_000_000, 64_000_000, 1_000_000_000,
                               2**31 - 2, 2**31 - 1])
def test_fast_mod_exhaustive(M):
    """Every hash value h in [0, p) reduced mod M on the device equals torch's
    remainder (a = 1, b = 0, T = C = Z = 1 makes the base exactly h mod M)."""
    dev = torch.device("cuda", 0)
    P = 2**31 - 1
    chunk = 1 << 28
    out = torch.empty(chunk, dtype=torch.int32, device=dev)
    for start in range(0, P, chunk):
        n = min(chunk, P - start)
        idx = torch.arange(start, start + n, dtype=torch.int64, device=dev)
        off = torch.tensor([0, n], dtype=torch.int64, device=dev)
        hp = pss.make_hash_params(a=1, b=0, num_tables=1, batch=1, num_indices=n)
        pss.pss_debug_addresses(M, 1, 1, hp, idx, off, out[:n])
        ok = torch.equal(out[:n].to(torch.int64), torch.remainder(idx, M))
        assert ok, f"mismatch in [{start}, {start + n}) for M={M}"
        del idx


def test_forward_integer_valued_bit_exact():
    """w[m] = m: every pooled sum is an integer below 2^24, so the GPU must
    reproduce the oracle bit for bit (pins addresses, wrap and pooling)."""
    rng = np.random.default_rng(11)
    wl = synth.get("c1").scaled(B=200, bag="poisson:12:0:64")
    w = np.arange(wl.M, dtype=np.float32)
    L = Layer(wl, w=w)
    got = L.forward()
    want = o.forward(w, wl.M, wl.Z, wl.d, wl.T, L.B, L.a, L.b, L.x.indices, L.x.offsets)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    del rng


@pytest.mark.parametrize("case", CASES, ids=_id)
def test_forward_parity(case):
    key, B, M = case
    L = Layer(synth.get(key), B=B, M=M)
    got = L.forward()
    ref, s_abs = L.ref_forward()
    parity.check_forward(got, ref, s_abs, 1e-5)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("case", CASES, ids=_id)
def test_backward_update_parity(case, variant):
    key, B, M = case
    L = Layer(synth.get(key), B=B, M=M, flags=VARIANTS[variant])
    g = synth.make_grad(L.wl, B=L.B)
    L.backward(g)
    w_ref, s_ref, G, A, cnt = L.ref_backward(g)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("key", ["c3", "c5"])
def test_adagrad_warm_state(key, variant):
    """Adagrad from s0 = 0.1: well conditioned everywhere, no exemptions."""
    L = Layer(synth.get(key), B=40, s0=0.1, flags=VARIANTS[variant])
    g = synth.make_grad(L.wl, B=L.B)
    L.backward(g)
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    ex = parity.check_update(L, L.weights(), L.state.cpu().numpy(), w_ref, s_ref, G, A, L.wl.lr)
    assert ex == 0


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("key,M,Z,d", [("c1", 4096, 4, 16), ("c1", 97, 8, 24), ("c3", 1000, 16, 64),
                                       ("c1", 300, 1, 7), ("c5", 5000, 128, 128)])
def test_unit_gradient_counts_bit_exact(key, M, Z, d, variant):
    """grad_out = 1, w = 0, lr = 1 ("loss = sum of retrieved elements"):
    w_new[m] = -(number of reads of m), an exact integer, wrap included."""
    wl = synth.get(key).scaled(M=M, Z=Z, d=d, optimizer="sgd", weight_dtype="f32")
    L = Layer(wl, B=150, w=np.zeros(M, dtype=np.float32), flags=VARIANTS[variant])
    ones = np.ones((L.B, wl.T * wl.d), dtype=np.float32)
    L.backward(ones, lr=1.0)
    _, _, _, _, cnt = L.ref_backward(ones, lr=1.0)
    assert np.array_equal(L.weights(), -cnt.astype(np.float32))


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_gradient_mass_per_chunk_offset(variant):
    """Masking grad_out to columns c with c mod Z = k moves exactly
    lr * (masked gradient mass) out of the array, for every k."""
    wl = synth.get("c1")
    for k in range(wl.Z):
        L = Layer(wl, B=256, flags=VARIANTS[variant])
        g = synth.make_grad(wl, B=L.B)
        cols = (np.arange(wl.T * wl.d) % wl.d) % wl.Z == k
        gk = np.where(cols[None, :], g, 0).astype(np.float32)
        L.backward(gk)
        moved = (L.w_host.astype(np.float64) - L.weights().astype(np.float64)).sum()
        lens = np.diff(L.x.offsets).reshape(wl.T, L.B)
        gk3 = gk.astype(np.float64).reshape(L.B, wl.T, wl.d)
        mass = sum(lens[t, b] * gk3[b, t].sum() for t in range(wl.T) for b in range(L.B))
        _, _, _, A, _ = L.ref_backward(gk)
        assert abs(moved - wl.lr * mass) <= 1e-5 * (np.abs(L.w_host).sum() + wl.lr * A.sum())


EDGE = [
    # (name, overrides, B)
    ("empty-and-long-bags", dict(bag="poisson:30:0:200"), 70),
    ("all-bags-empty", dict(bag="poisson:0:0:0"), 65),
    ("d48-z16", dict(d=48, Z=16), 90),
    ("d24-z3-wrap", dict(d=24, Z=3, M=61), 33),
    ("d640-z64-slabs", dict(d=640, Z=64), 20),
    ("d4096-z1024", dict(d=4096, Z=1024, M=5000), 3),
    ("Z-equals-M", dict(d=32, Z=32, M=32), 40),
    ("M-one", dict(d=4, Z=1, M=1), 40),
    ("one-table-one-bag", dict(T=1), 1),
]


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("name,over,B", EDGE, ids=[e[0] for e in EDGE])
@pytest.mark.parametrize("opt", ["sgd", "adagrad"])
def test_edge_shapes(name, over, B, opt, variant):
    wl = synth.get("c1").scaled(optimizer=opt, lr=0.05, **over)
    L = Layer(wl, B=B, flags=VARIANTS[variant])
    got = L.forward()
    ref, s_abs = L.ref_forward()
    parity.check_forward(got, ref, s_abs, 1e-5)
    assert np.array_equal(L.debug_bases().astype(np.uint64),
                          o.chunk_bases(wl.M, wl.Z, wl.d, wl.T, B, L.a, L.b, L.x.indices, L.x.offsets))
    g = synth.make_grad(wl, B=B)
    L.backward(g)
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, wl.lr)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_bf16_sgd_storage(variant):
    """bf16 storage with SGD goes through the gradient buffer and rounds once."""
    wl = synth.get("c5").scaled(optimizer="sgd", lr=0.1, M=300_000)
    L = Layer(wl, B=500, flags=VARIANTS[variant])
    g = synth.make_grad(wl, B=L.B)
    L.backward(g)
    w_ref, _, G, A, _ = L.ref_backward(g)
    parity.check_update(L, L.weights(), None, w_ref, None, G, A, wl.lr)


@pytest.mark.parametrize("key", ["c2", "c3"])
def test_sorted_and_atomic_agree(key):
    """Alg. 1's two branches compute the same gradient: the sorted (unique
    tokens, summed) and the per-contribution atomic deposits agree to the
    normalised tolerance element by element."""
    wl = synth.get(key).scaled(optimizer="adagrad", lr=0.01)
    La = Layer(wl, B=200, flags=pss.PSS_BWD_ATOMIC, s0=0.1)
    Ls = Layer(wl, B=200, flags=pss.PSS_BWD_SORTED, s0=0.1)
    g = synth.make_grad(wl, B=200)
    La.backward(g)
    Ls.backward(g)
    _, s_ref, G, A, _ = La.ref_backward(g)
    sa = La.state.cpu().numpy().astype(np.float64)
    ss = Ls.state.cpu().numpy().astype(np.float64)
    bound = 1e-5 * (0.1 + A * A) + 1e-30
    assert np.all(np.abs(sa - ss) <= 2 * bound)
    assert np.all(np.abs(ss - s_ref) <= bound)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("Z", [1, 32, 128])
def test_microbenchmark_shape_counts(Z, variant):
    """The paper's micro-benchmark shape: one table, batch 10240, d = 128,
    loss = sum of retrieved elements (grad_out = 1).  With w = 0 and lr = 1
    the update is minus the read count of every element, exactly."""
    wl = synth.get("c1").scaled(T=1, B=10240, d=128, Z=Z, M=128_000, cardinality="fixed:10000000",
                                optimizer="sgd", weight_dtype="f32")
    L = Layer(wl, w=np.zeros(wl.M, dtype=np.float32), flags=VARIANTS[variant])
    ones = np.ones((L.B, wl.d), dtype=np.float32)
    L.backward(ones, lr=1.0)
    _, _, _, _, cnt = L.ref_backward(ones, lr=1.0)
    assert np.array_equal(L.weights(), -cnt.astype(np.float32))


def _irregular_equal_count(wl, B, seed=5):
    """As many items as bags, but not one per bag: starting from one item per
    bag, 1500 items move between random bags inside bags [5000, 9000), which
    leaves the sort tiles before and after that range one-hot and the tiles
    inside it irregular (bags of 0 .. several items)."""
    nb = wl.T * B
    rng = np.random.default_rng(seed)
    lens = np.ones(nb, dtype=np.int64)
    lo, hi = min(5000, nb - 2), min(9000, nb)
    for _ in range(1500):
        i, j = rng.integers(lo, hi, 2)
        if lens[j] > 0 and i != j:
            lens[i] += 1
            lens[j] -= 1
    offsets = np.zeros(nb + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    assert offsets[-1] == nb
    card = int(wl.cardinality.split(":")[1]) if wl.cardinality.startswith("fixed") else 1000
    indices = rng.integers(0, card, nb, dtype=np.int64)
    return synth.Inputs(indices=indices, offsets=offsets, B=B)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("opt,mean", [("sgd", False), ("adagrad", True)])
def test_irregular_bags_with_one_item_per_bag_on_average(variant, opt, mean):
    """A batch with as many items as bags takes the one-hot paths (keygen in
    item space fused with the first radix histogram); tiles whose bags are
    not one item each fall back to finding each item's bag by search."""
    wl = synth.get("c2").scaled(optimizer=opt, lr=0.05, M=1_000_000)
    B = 700
    L = Layer(wl, B=B, flags=VARIANTS[variant], mean=mean, s0=0.1 if opt == "adagrad" else 0.0)
    L.x = _irregular_equal_count(wl, B)
    L.indices = torch.from_numpy(L.x.indices).to(L.dev)
    L.offsets = torch.from_numpy(L.x.offsets).to(L.dev)
    got = L.forward()
    ref, s_abs = L.ref_forward()
    parity.check_forward(got, ref, s_abs, 1e-5)
    g = synth.make_grad(wl, B=B)
    L.backward(g)
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, wl.lr)
