"""GPU parity: libzo's kernels against the CPU oracle on the same seeded inputs.

Bars: generated probe bits and perturb results bit-exact; update within
|gpu - oracle| <= 1e-6 * max(|theta|, lr * sum_k |c_k|) for fp32 weights, and for bf16
weights within one bf16 ulp of the result plus that same fp32 allowance (the kernel forms
theta - lr * sum in fp32 before its single rounding to bf16, so where the result cancels
to nearly zero the fp32 rounding of the operands can exceed a bf16 ulp of the result);
coefficients bit-exact (host tests).
"""

import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_38095_amd as zo
import workloads

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def note(msg):
    print(msg, flush=True)


def to_dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_spacing(x):
    m = np.abs(x)
    e = np.floor(np.log2(np.maximum(m, 2.0 ** -126)))
    return np.where(m < 2.0 ** -126, 2.0 ** -133, 2.0 ** (e - 7))


def assert_bf16_within_1ulp(got_bits, want_bits, theta_bits=None, c=(), lr=0.0):
    g = oracle.bf16_to_f64(got_bits)
    w = oracle.bf16_to_f64(want_bits)
    err = np.abs(g - w)
    allow = bf16_spacing(np.maximum(np.abs(g), np.abs(w)))
    if theta_bits is not None:
        scale = np.maximum(np.abs(oracle.bf16_to_f64(theta_bits)), abs(lr) * np.abs(np.asarray(c, np.float64)).sum())
        allow = allow + 1e-6 * scale
    ok = err <= allow
    assert np.all(ok), f"{np.count_nonzero(~ok)} elements beyond 1 bf16 ulp; first at {np.argmax(~ok)}"
    return np.count_nonzero(got_bits != want_bits)


def assert_f32_update_close(got, want, c, lr):
    scale = np.maximum(np.abs(want.astype(np.float64)), abs(lr) * np.abs(np.asarray(c, np.float64)).sum())
    err = np.abs(got.astype(np.float64) - want.astype(np.float64))
    ok = err <= 1e-6 * scale
    assert np.all(ok), f"max rel err {np.max(err / scale):.3e}"
    return float(np.max(err / scale))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    zo.library()
    zo.zo_set_max_blocks(0)
    yield
    zo.zo_set_max_blocks(0)


# ----------------------------------------------------------------------------- generator
@pytest.mark.parametrize("tile_begin,n_tiles,seed,step,group", [
    (0, 1, 0, 0, 0),
    (0, 4096, 1, 0, 0),
    (12345, 777, 2 ** 64 - 1, 2 ** 32 - 1, 3),
    (2 ** 32 - 5, 20, 0xDEADBEEFCAFEF00D, 7, 2 ** 29 - 1),   # counter word 0 wraps into word 1
    (1_873_342_080, 1000, 42, 1, 1),                         # OPT-30B's last tiles
])
def test_gen_bits_bit_exact(tile_begin, n_tiles, seed, step, group):
    note(f"gen_bits tiles [{tile_begin}, +{n_tiles}) seed {seed} step {step} group {group}")
    out = torch.zeros(16 * n_tiles, dtype=torch.uint8, device=DEV)
    zo.zo_gen_bits(out, tile_begin, seed, step, group)
    got = out.cpu().numpy().reshape(n_tiles, 16)
    np.testing.assert_array_equal(got, oracle.tile_bytes(tile_begin, n_tiles, seed, step, group))


# ----------------------------------------------------------------------------- perturb
PERTURB_CASES = [
    # n, offset, k, eps
    (1, 0, 0, 1e-3), (15, 0, 1, 1e-3), (16, 0, 7, -2e-3), (17, 0, 8, 1e-3), (1000, 3, 63, 1e-4),
    (65_536 + 13, 0, 1000, 1e-3), (4099, 2 ** 35 + 7, 5, -2e-3), (300_000, 16, 17, 1e-3),
    # the top of both index ranges: last global elements below 2^64, the last probe 2^32 - 1
    # (odd offsets take the element path, 2^64 - 2^17 the vector path)
    (5_000, 2 ** 64 - 5_001, 2 ** 32 - 1, 1e-3), (2 ** 17 - 1, 2 ** 64 - 2 ** 17, 2 ** 32 - 9, -2e-3),
]


def test_gen_bits_known_answer():
    """Tile 0, seed 0, step 0, group 0 is Philox4x32-10 on the all-zero counter and key: the
    block equals the published known-answer output (the other known-answer inputs lie outside
    the library's index range)."""
    golden = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "philox4x32_10_kat.txt")
    rows = [[int(x, 16) for x in ln.split()] for ln in open(golden) if ln.strip() and not ln.startswith("#")]
    want = np.array(rows[0][6:10], dtype=np.uint32)
    assert rows[0][:6] == [0] * 6
    out = torch.zeros(16, dtype=torch.uint8, device=DEV)
    zo.zo_gen_bits(out, 0, 0, 0, 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint32), want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,offset,k,eps", PERTURB_CASES)
def test_perturb_bit_exact(dtype, n, offset, k, eps):
    note(f"perturb {dtype} n {n} offset {offset} k {k} eps {eps}")
    seed, step = 1234567, 3
    if dtype == "f32":
        th = workloads.normal_f32(n, n)
        t = to_dev_f32(th)
        zo.zo_perturb(t, k, eps, seed, step, offset=offset)
        np.testing.assert_array_equal(t.cpu().numpy(), oracle.perturb(th, "f32", offset, seed, step, k, eps))
    else:
        th = workloads.normal_bf16_bits(n, n)
        t = to_dev_bf16(th)
        zo.zo_perturb(t, k, eps, seed, step, offset=offset)
        np.testing.assert_array_equal(host_bits(t), oracle.perturb(th, "bf16", offset, seed, step, k, eps))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shift,offset", [(1, 1), (1, 0), (3, 0), (5, 12)])
def test_perturb_unaligned_storage(dtype, shift, offset):
    """A view starting mid-tile: vector path when (pointer, offset) agree, element path otherwise."""
    note(f"perturb unaligned {dtype} shift {shift} offset {offset}")
    n = 5000
    if dtype == "f32":
        th = workloads.normal_f32(n + shift, 5)
        t = to_dev_f32(th)
        zo.zo_perturb(t[shift:], 9, 1e-3, 1, 2, offset=offset)
        want = th.copy()
        want[shift:] = oracle.perturb(th[shift:], "f32", offset, 1, 2, 9, 1e-3)
        np.testing.assert_array_equal(t.cpu().numpy(), want)
    else:
        th = workloads.normal_bf16_bits(n + shift, 5)
        t = to_dev_bf16(th)
        zo.zo_perturb(t[shift:], 9, 1e-3, 1, 2, offset=offset)
        want = th.copy()
        want[shift:] = oracle.perturb(th[shift:], "bf16", offset, 1, 2, 9, 1e-3)
        np.testing.assert_array_equal(host_bits(t), want)


def test_perturb_bf16_rounding_ties_and_subnormals():
    """Crafted exact ties of the fp32 sum (both parities) and subnormal bf16 weights."""
    vals = []
    for m in range(128):
        vals += [1.0 + m * 2.0 ** -7, -(1.0 + m * 2.0 ** -7), 0.5 + m * 2.0 ** -8]
    th = oracle.f32_to_bf16(np.array(vals, np.float32))
    sub = np.arange(1, 200, dtype=np.uint16)  # positive bf16 subnormals
    th = np.concatenate([th, sub, sub | np.uint16(0x8000), np.zeros(7, np.uint16)])
    for eps in (2.0 ** -8, 2.0 ** -9, 3 * 2.0 ** -130, 1e-3):
        t = to_dev_bf16(th)
        zo.zo_perturb(t, 3, eps, 77, 0)
        np.testing.assert_array_equal(host_bits(t), oracle.perturb(th, "bf16", 0, 77, 0, 3, eps))


SPECIALS = [0.0, -0.0, np.inf, -np.inf, np.nan, 3.3895314e38, -3.3895314e38, 1e-40, -1e-40, 1.1754944e-38, 1.0]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("eps", [1e-3, 0.0, 3e38])
def test_special_values_match_oracle(dtype, eps):
    """Signed zeros, infinities, NaN, the largest finite values (overflow to inf), subnormals;
    eps = 0 leaves finite weights unchanged. NaN is compared as NaN (its payload is not fixed)."""
    n = 16 * 12 + 5
    vals = np.array((SPECIALS * (n // len(SPECIALS) + 1))[:n], dtype=np.float32)
    th = vals if dtype == "f32" else oracle.f32_to_bf16(vals)
    t = to_dev_f32(th) if dtype == "f32" else to_dev_bf16(th)
    zo.zo_perturb(t, 2, eps, 4, 4)
    want = oracle.perturb(th, dtype, 0, 4, 4, 2, eps)
    got = t.cpu().numpy() if dtype == "f32" else host_bits(t)
    gf = got.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(got)
    wf = want.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(want)
    assert np.array_equal(np.isnan(gf), np.isnan(wf))
    ok = ~np.isnan(wf)
    np.testing.assert_array_equal(got[ok], want[ok])
    c = np.array([0.5, -0.25], np.float32)
    zo.zo_update(t, c, 1e-3, 4, 4)
    u_want = oracle.update(want, dtype, 0, 4, 4, c, 1e-3)
    u_got = t.cpu().numpy() if dtype == "f32" else host_bits(t)
    uf = u_got.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(u_got)
    wf = u_want.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(u_want)
    assert np.array_equal(np.isnan(uf), np.isnan(wf))
    fin = np.isfinite(wf)
    assert np.array_equal(uf[~fin & ~np.isnan(wf)], wf[~fin & ~np.isnan(wf)])  # infinities agree
    err = np.abs(uf[fin] - wf[fin])
    assert np.all(err <= 1e-6 * np.maximum(np.abs(wf[fin]), 1e-3 * 0.75) + (0 if dtype == "f32" else bf16_spacing(np.abs(wf[fin]))))


def test_perturb_schedule_restores_fp32_within_1ulp():
    """Algorithm 1's +eps, -2 eps, +eps on the tiny workload: within 1 ulp of the largest intermediate."""
    th = workloads.tiny_theta()
    t = to_dev_f32(th)
    mags = [np.abs(th)]
    for e in (1e-3, -2e-3, 1e-3):
        zo.zo_perturb(t, 2, e, 0, 0)
        mags.append(np.abs(t.cpu().numpy()))
    got = t.cpu().numpy()
    M = np.maximum.reduce(mags)
    assert np.all(np.abs(got.astype(np.float64) - th) <= np.spacing(M).astype(np.float64))


# ----------------------------------------------------------------------------- update
UPDATE_CASES = [
    # n, offset, k_base, K
    (1000, 0, 0, 1), (4096, 0, 0, 4), (4097, 0, 0, 8), (3333, 5, 0, 9), (70_001, 0, 0, 16),
    (20_000, 2 ** 33 + 1, 0, 24), (20_000, 0, 0, 32), (50_000, 0, 0, 64), (9_000, 0, 0, 65),
    (5_000, 0, 0, 200), (3_000, 0, 0, 256), (10_000, 48, 3, 16), (10_000, 0, 8, 16), (7_000, 0, 100, 57),
    (4_100, 0, 0, 512), (3_000, 17, 0, 1024), (2_500, 0, 5, 1024),
    (6_000, 2 ** 64 - 6_001, 2 ** 32 - 40, 40), (5_000, 2 ** 60, 2 ** 32 - 64, 64),
    (2 ** 17 - 1, 2 ** 64 - 2 ** 17, 2 ** 32 - 24, 24),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,offset,k_base,K", UPDATE_CASES)
def test_update_matches_oracle(dtype, n, offset, k_base, K):
    note(f"update {dtype} n {n} offset {offset} k_base {k_base} K {K}")
    seed, step, lr = 99, 5, 1e-3
    c = np.random.default_rng(K).standard_normal(K).astype(np.float32) * 3
    if dtype == "f32":
        th = workloads.normal_f32(n, 1)
        t = to_dev_f32(th)
        zo.zo_update_ex(t, c, lr, seed, step, offset=offset, k_base=k_base)
        want = oracle.update(th, "f32", offset, seed, step, c, lr, k_base=k_base)
        assert_f32_update_close(t.cpu().numpy(), want, c, lr)
    else:
        th = workloads.normal_bf16_bits(n, 1)
        t = to_dev_bf16(th)
        zo.zo_update_ex(t, c, lr, seed, step, offset=offset, k_base=k_base)
        want = oracle.update(th, "bf16", offset, seed, step, c, lr, k_base=k_base)
        assert_bf16_within_1ulp(host_bits(t), want, th, c, lr)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_update_k1_equals_perturb(dtype):
    n, c0, lr = 100_003, np.float32(0.7310586), np.float32(1e-3)
    base = workloads.normal_f32(n, 8)
    if dtype == "f32":
        a, b = to_dev_f32(base), to_dev_f32(base)
    else:
        bits = oracle.f32_to_bf16(base)
        a, b = to_dev_bf16(bits), to_dev_bf16(bits)
    zo.zo_update(a, [c0], lr, 4, 2)
    zo.zo_perturb(b, 0, -(lr * c0), 4, 2)
    assert torch.equal(a.view(torch.int16) if dtype == "bf16" else a, b.view(torch.int16) if dtype == "bf16" else b)


@pytest.mark.parametrize("op", ["perturb", "update16", "update64", "update200"])
def test_results_independent_of_grid(op):
    n = 1_000_003
    th = workloads.normal_bf16_bits(n, 3)
    c = np.random.default_rng(0).standard_normal(256).astype(np.float32)
    outs = []
    for blocks in (1, 7, 64, 0):
        zo.zo_set_max_blocks(blocks)
        t = to_dev_bf16(th)
        if op == "perturb":
            zo.zo_perturb(t, 11, 1e-3, 5, 1)
        else:
            K = int(op[6:])
            zo.zo_update(t, c[:K], 1e-3, 5, 1)
        outs.append(host_bits(t))
    zo.zo_set_max_blocks(0)
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])


def test_update_linearity_fp32():
    th = workloads.normal_f32(200_000, 4)
    c = np.random.default_rng(9).standard_normal(16).astype(np.float32)
    t = to_dev_f32(th)
    zo.zo_update(t, c, 1e-3, 1, 1)
    mid = np.abs(t.cpu().numpy())
    zo.zo_update(t, -c, 1e-3, 1, 1)
    got = t.cpu().numpy().astype(np.float64)
    M = np.maximum(np.abs(th), mid)
    assert np.all(np.abs(got - th) <= 2 * np.spacing(M).astype(np.float64))


def test_empty_and_noop_calls():
    t = torch.zeros(0, dtype=torch.float32, device=DEV)
    zo.zo_perturb(t, 0, 1e-3, 0, 0)
    zo.zo_update(t, [1.0], 1e-3, 0, 0)
    u = to_dev_f32(workloads.normal_f32(100, 0))
    before = u.clone()
    zo.zo_update(u, [], 1e-3, 0, 0)
    assert torch.equal(u, before)
    with pytest.raises(zo.ZoError):
        zo.zo_update(u, np.zeros(zo.ZO_K_MAX + 1, np.float32), 1e-3, 0, 0)
    side = torch.cuda.Stream()
    zo.zo_perturb_segments([], [], 0, 1e-3, 0, 0.0, 0, 0, stream=side)  # an empty list on a given stream
    zo.zo_update_segments([], [], [1.0], 1e-3, 0, 0, stream=side)
    zo.zo_perturb_segments([u[:0]], [0], 0, 1e-3, 0, 0.0, 0, 0)  # an empty tensor
    torch.cuda.synchronize()
    assert torch.equal(u, before)


# ----------------------------------------------------------------------------- fused transitions
PERTURB2_CASES = [
    # n, offset, k_a, e_a, k_b, e_b
    (1000, 0, 3, 1e-3, 4, 1e-3), (70_001, 0, 7, 1e-3, 8, 1e-3), (4099, 2 ** 35 + 7, 0, 1e-3, 1, 1e-3),
    (5000, 3, 5, 1e-3, 5, 1e-3), (5000, 0, 5, 1e-3, 5, -1e-3), (20_000, 0, 9, 1e-3, 100, -3.7e-4),
    (3000, 16, 2, -2e-3, 2, 0.0), (17, 0, 1, 1e-3, 2, 1e-3),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,offset,k_a,e_a,k_b,e_b", PERTURB2_CASES)
def test_perturb2_bit_exact(dtype, n, offset, k_a, e_a, k_b, e_b):
    note(f"perturb2 {dtype} n {n} offset {offset} ({k_a}, {e_a}) ({k_b}, {e_b})")
    seed, step = 77, 9
    if dtype == "f32":
        th = workloads.normal_f32(n, 2)
        t = to_dev_f32(th)
        zo.zo_perturb2(t, k_a, e_a, k_b, e_b, seed, step, offset=offset)
        want = oracle.perturb2(th, "f32", offset, seed, step, k_a, e_a, k_b, e_b)
        np.testing.assert_array_equal(t.cpu().numpy(), want)
    else:
        th = workloads.normal_bf16_bits(n, 2)
        t = to_dev_bf16(th)
        zo.zo_perturb2(t, k_a, e_a, k_b, e_b, seed, step, offset=offset)
        np.testing.assert_array_equal(host_bits(t), oracle.perturb2(th, "bf16", offset, seed, step, k_a, e_a, k_b, e_b))


def test_perturb2_zero_second_scale_equals_perturb():
    bits = workloads.normal_bf16_bits(100_003, 3)
    a, b = to_dev_bf16(bits), to_dev_bf16(bits)
    zo.zo_perturb2(a, 6, 1e-3, 13, 0.0, 5, 5)
    zo.zo_perturb(b, 6, 1e-3, 5, 5)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def assert_restore_update_close(got, want, theta, c, lr, er, dtype):
    th64 = theta.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(theta)
    g64 = got.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(got)
    w64 = want.astype(np.float64) if dtype == "f32" else oracle.bf16_to_f64(want)
    scale = np.maximum(np.maximum(np.abs(th64) + abs(er), np.abs(w64)), abs(lr) * np.abs(np.asarray(c, np.float64)).sum())
    allow = 1e-6 * scale
    if dtype == "bf16":
        allow = allow + bf16_spacing(np.maximum(np.abs(g64), np.abs(w64)))
    err = np.abs(g64 - w64)
    assert np.all(err <= allow), f"{np.count_nonzero(err > allow)} elements out of bound"


RESTORE_CASES = [
    # n, offset, k_base, K, k_restore
    (50_000, 0, 0, 16, 15), (20_000, 5, 0, 4, 3), (30_000, 0, 0, 64, 63), (9_000, 2 ** 33, 0, 200, 199),
    (10_000, 0, 0, 16, 40), (10_000, 0, 8, 16, 0), (7_000, 0, 3, 13, 15), (5_000, 0, 0, 0, 2),
    # restore probe inside the update's groups but not in the last one (its words are generated
    # again rather than taken from the group sum)
    (12_000, 0, 0, 16, 3), (12_000, 17, 0, 32, 9), (6_000, 0, 0, 64, 50),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,offset,k_base,K,k_restore", RESTORE_CASES)
def test_update_restore_matches_oracle(dtype, n, offset, k_base, K, k_restore):
    note(f"update_restore {dtype} n {n} offset {offset} k_base {k_base} K {K} restore {k_restore}")
    seed, step, lr, er = 31, 4, 1e-3, 1e-3
    c = np.random.default_rng(K + 1).standard_normal(K).astype(np.float32) * 3
    th = workloads.normal_f32(n, 3) if dtype == "f32" else workloads.normal_bf16_bits(n, 3)
    t = to_dev_f32(th) if dtype == "f32" else to_dev_bf16(th)
    zo.zo_update_restore(t, c, lr, seed, step, k_restore, er, offset=offset, k_base=k_base)
    got = t.cpu().numpy() if dtype == "f32" else host_bits(t)
    want = oracle.update_restore(th, dtype, offset, seed, step, c, lr, k_restore, er, k_base=k_base)
    assert_restore_update_close(got, want, th, c, lr, er, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_update_restore_zero_restore_equals_update(dtype):
    base = workloads.normal_f32(100_003, 4)
    c = np.random.default_rng(2).standard_normal(16).astype(np.float32)
    if dtype == "f32":
        a, b = to_dev_f32(base), to_dev_f32(base)
    else:
        bits = oracle.f32_to_bf16(base)
        a, b = to_dev_bf16(bits), to_dev_bf16(bits)
    zo.zo_update_restore(a, c, 1e-3, 6, 6, 15, 0.0)
    zo.zo_update(b, c, 1e-3, 6, 6)
    view = (lambda x: x.view(torch.int16)) if dtype == "bf16" else (lambda x: x)
    assert torch.equal(view(a), view(b))


def test_full_tiny_step_fused():
    """The tiny workload in 2K + 1 sweeps: +eps z_0; per probe -2 eps z_k then the merged
    restore / next +eps; the last restore merged with the update."""
    w = workloads.WORKLOADS["tiny"]
    K = w.K[0]
    th = workloads.tiny_theta(w.n)
    lp, lm, l0 = workloads.synthetic_losses(K, 1)
    t = to_dev_f32(th)
    zo.zo_perturb(t, 0, w.eps, 0, 0)
    for k in range(K):
        zo.zo_perturb(t, k, -2 * w.eps, 0, 0)
        if k + 1 < K:
            zo.zo_perturb2(t, k, w.eps, k + 1, w.eps, 0, 0)
    c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
    zo.zo_update_restore(t, c, w.lr, 0, 0, K - 1, w.eps)
    want, co, _ = oracle.full_step_fused(th, "f32", 0, 0, 0, w.eps, w.lr, lp, lm, l0)
    np.testing.assert_array_equal(c, co["c"])
    assert_f32_update_close(t.cpu().numpy(), want, c, w.lr)


# ----------------------------------------------------------------------------- separate tensors
def _model_tensors(dtype, sizes, seed):
    """Separate device tensors (one allocation each) plus their global offsets in a flat layout."""
    offs, o, ts, host = [], 0, [], []
    for i, sz in enumerate(sizes):
        h = workloads.normal_f32(sz, seed + i) if dtype == "f32" else workloads.normal_bf16_bits(sz, seed + i)
        host.append(h)
        ts.append(to_dev_f32(h) if dtype == "f32" else to_dev_bf16(h))
        offs.append(o)
        o += sz
    return ts, offs, host


SEG_SIZES = [5120 * 3 + 7, 5120, 5120, 16, 1, 0, 3000, 20_480 * 5, 5120, 2048, 4096 + 3]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_segments_match_flat_and_oracle(dtype):
    """Each tensor of a segment list gets exactly what the oracle (and the flat call) gives it."""
    ts, offs, host = _model_tensors(dtype, SEG_SIZES, 10)
    seed, step, eps = 5, 2, 1e-3
    c = np.random.default_rng(3).standard_normal(16).astype(np.float32)
    get = (lambda t: t.cpu().numpy()) if dtype == "f32" else host_bits
    zo.zo_perturb_segments(ts, offs, 3, eps, 0, 0.0, seed, step)
    for t, o, h in zip(ts, offs, host):
        np.testing.assert_array_equal(get(t), oracle.perturb(h, dtype, o, seed, step, 3, eps))
    mid = [get(t) for t in ts]
    zo.zo_perturb_segments(ts, offs, 3, eps, 4, eps, seed, step)
    for t, o, m in zip(ts, offs, mid):
        np.testing.assert_array_equal(get(t), oracle.perturb2(m, dtype, o, seed, step, 3, eps, 4, eps))
    mid = [get(t) for t in ts]
    # flat reference: the same values in one buffer, swept by the single-tensor call
    flat_h = np.concatenate(mid)
    flat = to_dev_f32(flat_h) if dtype == "f32" else to_dev_bf16(flat_h)
    zo.zo_update_restore(flat, c, 1e-3, seed, step, 4, eps)
    zo.zo_update_segments(ts, offs, c, 1e-3, seed, step, k_restore=4, eps_restore=eps)
    flat_out = get(flat)
    for t, o, m in zip(ts, offs, mid):
        got = get(t)
        np.testing.assert_array_equal(got, flat_out[o:o + m.size])
        assert_restore_update_close(got, oracle.update_restore(m, dtype, o, seed, step, c, 1e-3, 4, eps), m, c,
                                    1e-3, eps, dtype)


def test_segments_many_launches_and_unaligned_views():
    """150 tensors (three batched launches), some of them views that start mid-vector, in a
    shuffled global order."""
    rng = np.random.default_rng(4)
    sizes = [int(s) for s in rng.integers(1, 9000, 150)]
    base = [workloads.normal_bf16_bits(s + 3, 100 + i) for i, s in enumerate(sizes)]
    owners = [to_dev_bf16(b) for b in base]
    shifts = [int(x) for x in rng.integers(0, 4, 150)]
    ts = [own[sh:sh + s] for own, sh, s in zip(owners, shifts, sizes)]
    order = rng.permutation(150)
    offs, o = [0] * 150, 7
    for i in order:
        offs[i] = o
        o += sizes[i] + int(rng.integers(0, 40))
    before = [host_bits(t) for t in ts]
    c = rng.standard_normal(24).astype(np.float32)
    zo.zo_perturb_segments(ts, offs, 9, 1e-3, 0, 0.0, 8, 8)
    zo.zo_update_segments(ts, offs, c, 1e-3, 8, 8)
    for t, own, sh, s, o_, b, orig in zip(ts, owners, shifts, sizes, offs, before, base):
        p = oracle.perturb(b, "bf16", o_, 8, 8, 9, 1e-3)
        assert_bf16_within_1ulp(host_bits(t), oracle.update(p, "bf16", o_, 8, 8, c, 1e-3), p, c, 1e-3)
        full = host_bits(own)  # memory outside the view is untouched
        np.testing.assert_array_equal(full[:sh], orig[:sh])
        np.testing.assert_array_equal(full[sh + s:], orig[sh + s:])


def test_segments_equal_flat_bits_for_update():
    """The update over separate tensors is bit-identical to the update of the same flat buffer."""
    ts, offs, host = _model_tensors("bf16", SEG_SIZES, 30)
    flat = to_dev_bf16(np.concatenate(host))
    c = np.random.default_rng(5).standard_normal(64).astype(np.float32)
    zo.zo_update_segments(ts, offs, c, 1e-3, 1, 1)
    zo.zo_update(flat, c, 1e-3, 1, 1)
    flat_out = host_bits(flat)
    for t, o, h in zip(ts, offs, host):
        np.testing.assert_array_equal(host_bits(t), flat_out[o:o + h.size])


def test_segments_streaming_shape_equal_flat_bits():
    """Above the 256 MiB streaming threshold: 56 separately allocated tensors of ragged sizes
    (tiny ones among multi-million ones, none a multiple of the 32 KiB chunk, the first at a
    global offset of 777) get, in every element, the bits that the single-buffer calls give
    the same values laid out flat: perturb, a two-probe transition, the update and the update
    with restore at K = 16 (two waves per stream, one chunk per stream), K = 32 (two-plane
    32-copy tables in 1024-thread workgroups; 16-copy tables at two workgroups per CU) and
    K = 64 (16-copy tables shared by 1024 or 512 threads). The single-buffer calls are
    themselves checked against the oracle at full size."""
    rng = np.random.default_rng(13)
    sizes = [int(x) for x in rng.integers(1, 8_000_000, 50)] + [1, 7, 1023, 1024, 1025, 16_385]
    sizes = [sizes[i] for i in rng.permutation(len(sizes))]
    total, base = sum(sizes), 777
    assert 2 * total >= 256 << 20
    note(f"segments at streaming scale: {len(sizes)} tensors, {total} weights")
    flat = torch.empty(total, dtype=torch.bfloat16, device=DEV)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(14)
    flat.normal_(0.0, 0.02, generator=gen)
    starts = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
    ts = [flat[int(a):int(a) + sz].clone() for a, sz in zip(starts, sizes)]
    offs = [base + int(a) for a in starts]
    seed, step, eps, lr = 31, 4, 1e-3, 1e-3
    c16 = rng.standard_normal(16).astype(np.float32)
    c64 = rng.standard_normal(64).astype(np.float32)
    c32 = rng.standard_normal(32).astype(np.float32)

    def same(what):
        torch.cuda.synchronize()
        for i, (t, a, sz) in enumerate(zip(ts, starts, sizes)):
            assert torch.equal(t.view(torch.int16), flat[int(a):int(a) + sz].view(torch.int16)), f"{what}: tensor {i}"

    zo.zo_perturb(flat, 3, eps, seed, step, offset=base)
    zo.zo_perturb_segments(ts, offs, 3, eps, 0, 0.0, seed, step)
    same("perturb")
    zo.zo_perturb2(flat, 3, -2 * eps, 12, eps, seed, step, offset=base)
    zo.zo_perturb_segments(ts, offs, 3, -2 * eps, 12, eps, seed, step)
    same("perturb2")
    zo.zo_update_ex(flat, c16, lr, seed, step, offset=base)
    zo.zo_update_segments(ts, offs, c16, lr, seed, step)
    same("update K=16")
    zo.zo_update_restore(flat, c16, lr, seed, step, 12, -eps, offset=base)
    zo.zo_update_segments(ts, offs, c16, lr, seed, step, 12, -eps)
    same("update_restore K=16")
    zo.zo_update_ex(flat, c32, lr, seed, step, offset=base)
    zo.zo_update_segments(ts, offs, c32, lr, seed, step)
    same("update K=32")
    zo.zo_update_restore(flat, c32, lr, seed, step, 31, -eps, offset=base)
    zo.zo_update_segments(ts, offs, c32, lr, seed, step, 31, -eps)
    same("update_restore K=32")
    zo.zo_update_ex(flat, c64, lr, seed, step, offset=base)
    zo.zo_update_segments(ts, offs, c64, lr, seed, step)
    same("update K=64")
    zo.zo_update_restore(flat, c64, lr, seed, step, 63, -eps, offset=base)
    zo.zo_update_segments(ts, offs, c64, lr, seed, step, 63, -eps)
    same("update_restore K=64")


@pytest.mark.parametrize("op", ["perturb", "update16", "restore16", "update32", "restore32", "update64", "restore64"])
def test_streaming_results_independent_of_grid(op):
    """Above the streaming threshold, where the launches use two waves per stream, one or four
    chunks per stream and 512- or 1024-thread workgroups: capping the grid at 1, 7 or 300
    workgroups (every stream then loops over many chunks) leaves every bit of the result as
    the default grid gives it."""
    n = 144_000_019
    note(f"streaming grid independence: {op}")
    src = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(21)
    src.normal_(0.0, 0.02, generator=gen)
    c = np.random.default_rng(5).standard_normal(64).astype(np.float32)
    outs = []
    try:
        for blocks in (0, 1, 7, 300):
            zo.zo_set_max_blocks(blocks)
            t = src.clone()
            if op == "perturb":
                zo.zo_perturb(t, 11, 1e-3, 5, 1, offset=33)
            else:
                K = int(op[-2:])
                if op.startswith("update"):
                    zo.zo_update_ex(t, c[:K], 1e-3, 5, 1, offset=33)
                else:
                    zo.zo_update_restore(t, c[:K], 1e-3, 5, 1, K - 1, 1e-3, offset=33)
            torch.cuda.synchronize()
            outs.append(t)
    finally:
        zo.zo_set_max_blocks(0)
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))


def test_concurrent_streams_on_disjoint_tensors():
    """Calls on two streams over disjoint tensors run concurrently and give the serial results."""
    a_h = workloads.normal_bf16_bits(3_000_017, 20)
    b_h = workloads.normal_bf16_bits(2_000_003, 21)
    a, b = to_dev_bf16(a_h), to_dev_bf16(b_h)
    c = np.random.default_rng(6).standard_normal(16).astype(np.float32)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for it in range(3):
        zo.zo_perturb(a, it, 1e-3, 1, 1, stream=s1)
        zo.zo_perturb(b, it, -2e-3, 2, 1, stream=s2)
    zo.zo_update(a, c, 1e-3, 1, 1, stream=s1)
    zo.zo_update_ex(b, c[:8], 1e-3, 2, 1, offset=5, stream=s2)
    torch.cuda.synchronize()
    wa, wb = a_h, b_h
    for it in range(3):
        wa = oracle.perturb(wa, "bf16", 0, 1, 1, it, 1e-3)
        wb = oracle.perturb(wb, "bf16", 0, 2, 1, it, -2e-3)
    assert_bf16_within_1ulp(host_bits(a), oracle.update(wa, "bf16", 0, 1, 1, c, 1e-3), wa, c, 1e-3)
    assert_bf16_within_1ulp(host_bits(b), oracle.update(wb, "bf16", 5, 2, 1, c[:8], 1e-3), wb, c[:8], 1e-3)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_graph_capture_replays_match_eager(dtype):
    """A fused two-probe step captured into a HIP graph (through torch) and replayed three times,
    with eager work and synchronisations between the replays, equals the same calls applied
    eagerly the same number of times, bit for bit (the library records only kernel launches)."""
    n = 300_007
    if dtype == "f32":
        h = workloads.normal_f32(n, 30)
        a, g = torch.from_numpy(h).to(DEV), torch.from_numpy(h).to(DEV)
    else:
        h = workloads.normal_bf16_bits(n, 30)
        a, g = to_dev_bf16(h), to_dev_bf16(h)
    c = np.random.default_rng(8).standard_normal(2).astype(np.float32)
    eps, lr, seed, step = 1e-3, 1e-3, 77, 4

    def fused_step(t):
        zo.zo_perturb(t, 0, eps, seed, step)
        zo.zo_perturb(t, 0, -2 * eps, seed, step)
        zo.zo_perturb2(t, 0, eps, 1, eps, seed, step)
        zo.zo_perturb(t, 1, -2 * eps, seed, step)
        zo.zo_update_restore(t, c, lr, seed, step, 1, eps)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        fused_step(g)
    torch.cuda.synchronize()
    bits = (lambda t: t.cpu().numpy().view(np.uint32)) if dtype == "f32" else host_bits
    np.testing.assert_array_equal(bits(g), bits(a))  # capture launches nothing
    scratch = torch.ones(1 << 16, device=DEV)
    for replay in range(3):
        fused_step(a)
        graph.replay()
        scratch.mul_(1.5)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(bits(g), bits(a), err_msg=f"replay {replay}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sharded_calls_equal_the_full_buffer(dtype):
    """The element-range sharding of a model too large for one device: each shard is stepped
    by its own calls with its global offset (uneven cuts, some mid-tile and mid-chunk), and the
    concatenation equals the full-buffer calls bit for bit (perturb, two-probe transition,
    update with restore)."""
    n = 1_000_003
    cuts = [0, 123_457, 123_460, 600_001, n]
    h = workloads.normal_f32(n, 40) if dtype == "f32" else workloads.normal_bf16_bits(n, 40)
    dev = (lambda x: torch.from_numpy(x).to(DEV)) if dtype == "f32" else to_dev_bf16
    full, sharded = dev(h), dev(h)
    c = np.random.default_rng(9).standard_normal(24).astype(np.float32)
    seed, step, eps, lr = 5, 2, 1e-3, 1e-3
    zo.zo_perturb(full, 3, eps, seed, step)
    zo.zo_perturb2(full, 3, -2 * eps, 4, eps, seed, step)
    zo.zo_update_restore(full, c, lr, seed, step, 4, -eps)
    for a, b in zip(cuts, cuts[1:]):
        shard = sharded[a:b]
        zo.zo_perturb(shard, 3, eps, seed, step, offset=a)
        zo.zo_perturb2(shard, 3, -2 * eps, 4, eps, seed, step, offset=a)
        zo.zo_update_restore(shard, c, lr, seed, step, 4, -eps, offset=a)
    torch.cuda.synchronize()
    bits = (lambda t: t.cpu().numpy().view(np.uint32)) if dtype == "f32" else host_bits
    np.testing.assert_array_equal(bits(sharded), bits(full))


# ----------------------------------------------------------------------------- full step
def test_full_tiny_step():
    """The tiny fp32 workload: 2^20 weights, K = 4, eps 1e-3, lr 1e-4 (schedule + coeffs + update)."""
    w = workloads.WORKLOADS["tiny"]
    K = w.K[0]
    th = workloads.tiny_theta(w.n)
    lp, lm, l0 = workloads.synthetic_losses(K, 1)
    t = to_dev_f32(th)
    for k in range(K):
        for e in (w.eps, -2 * w.eps, w.eps):
            zo.zo_perturb(t, k, e, 0, 0)
    c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
    zo.zo_update(t, c, w.lr, 0, 0)
    want, co = oracle.full_step(th, "f32", 0, 0, 0, w.eps, w.lr, lp, lm, l0)
    np.testing.assert_array_equal(c, co["c"])
    assert_f32_update_close(t.cpu().numpy(), want, c, w.lr)


# ----------------------------------------------------------------------------- full size
def _windows(n, rng, count, size, boundaries=()):
    starts = [0, n - size, n - 37] + [int(b) - size // 2 for b in boundaries]
    starts += [int(s) for s in rng.integers(0, n - size, count)]
    return sorted({min(max(s, 0), n - 1) for s in starts})


@pytest.mark.parametrize("name,K", [("opt125m", 16), ("opt13b", 16), ("opt1.3b", 64), ("opt30b", 8), ("opt30b", 32),
                                    ("qwen3-1.7b", 60), ("qwen3-8b", 60)])
def test_full_size_sampled_windows(name, K):
    """At the full OPT-shaped size, in the benchmark's launch configuration, on 32 random
    windows of 2^20 weights plus the first window, the last (with the ragged tail) and windows
    across tensor boundaries: one perturb and one two-probe transition checked bit for bit on
    every window; the update and the update-with-restore checked on the first and last 2^15
    weights of every window (the oracle's K-probe sums are the slow part)."""
    w = workloads.WORKLOADS[name]
    n = w.n
    note(f"full-size {name}: n {n} K {K}")
    buf = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    workloads.fill_model_buffer_device(buf, w)
    rng = np.random.default_rng(7)
    offs = [o for _, o, _ in workloads.tensor_offsets(w)]
    bounds = [offs[1], offs[2], offs[len(offs) // 2], offs[-2]]
    size, part = 1 << 20, 1 << 15
    wins = _windows(n, rng, 32, size, bounds)
    assert len(wins) >= 32
    grab = lambda: [host_bits(buf[s:min(s + size, n)]) for s in wins]
    seed, step = 2024, 3
    before = grab()
    zo.zo_perturb(buf, 5, w.eps, seed, step)
    mid = grab()
    lp, lm, l0 = workloads.synthetic_losses(K, step)
    c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
    zo.zo_update(buf, c, w.lr, seed, step)
    after = grab()
    zo.zo_perturb2(buf, 5, w.eps, 6, w.eps, seed, step)
    trans = grab()
    zo.zo_update_restore(buf, c, w.lr, seed, step, 6, w.eps)
    final = grab()
    torch.cuda.synchronize()
    del buf
    torch.cuda.empty_cache()
    for s, b, m, a, tr, f in zip(wins, before, mid, after, trans, final):
        np.testing.assert_array_equal(m, oracle.perturb(b, "bf16", s, seed, step, 5, w.eps))
        np.testing.assert_array_equal(tr, oracle.perturb2(a, "bf16", s, seed, step, 5, w.eps, 6, w.eps))
        m_len = len(m)
        for lo in sorted({0, max(m_len - part, 0)}):
            hi = min(lo + part, m_len)
            g = s + lo
            assert_bf16_within_1ulp(a[lo:hi], oracle.update(m[lo:hi], "bf16", g, seed, step, c, w.lr),
                                    m[lo:hi], c, w.lr)
            assert_restore_update_close(f[lo:hi],
                                        oracle.update_restore(tr[lo:hi], "bf16", g, seed, step, c, w.lr, 6, w.eps),
                                        tr[lo:hi], c, w.lr, w.eps, "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("K", [8, 16, 24, 32, 48, 64])
def test_streaming_shapes_sampled_windows(dtype, K):
    """Every launch shape the library picks above the 256 MiB streaming threshold (perturb with
    one probe, two probes in one group and in two groups, update and update-with-restore with
    1 to 8 probe groups: spread or shared tables, 1-4 workgroups per CU or full occupancy, one
    or two groups in flight), for bf16 and fp32, on a ragged 288 MB buffer at global offset
    777: ten windows of 2^15 weights (the first, the last with the ragged tail, eight at random
    offsets) checked against the oracle after every sweep."""
    n = (144_000_019 if dtype == "bf16" else 72_000_011)
    off, seed, step, eps, lr = 777, 41, 6, 1e-3, 1e-3
    note(f"streaming shapes: {dtype} n {n} K {K}")
    t = torch.empty(n, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device=DEV)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(43)
    t.normal_(0.0, 0.02, generator=gen)
    size = 1 << 15
    rng = np.random.default_rng(K)
    wins = sorted({0, n - size} | {int(x) for x in rng.integers(0, n - size, 8)})
    if dtype == "bf16":
        grab = lambda: [host_bits(t[s:s + size]) for s in wins]
    else:
        grab = lambda: [t[s:s + size].cpu().numpy() for s in wins]
    c = rng.standard_normal(K).astype(np.float32)
    kr = K - 1  # restore probe inside the update's last group
    states = [grab()]
    zo.zo_perturb(t, 3, eps, seed, step, offset=off)
    states.append(grab())
    zo.zo_perturb2(t, 3, -2 * eps, 4, eps, seed, step, offset=off)  # one probe group
    states.append(grab())
    zo.zo_perturb2(t, 4, eps, 12, eps, seed, step, offset=off)  # two probe groups
    states.append(grab())
    zo.zo_update_ex(t, c, lr, seed, step, offset=off)
    states.append(grab())
    zo.zo_update_restore(t, c, lr, seed, step, kr, eps, offset=off)
    states.append(grab())
    torch.cuda.synchronize()
    del t
    torch.cuda.empty_cache()
    for i, s in enumerate(wins):
        b, p1, p2, p3, u, ur = (st[i] for st in states)
        g = off + s
        np.testing.assert_array_equal(p1, oracle.perturb(b, dtype, g, seed, step, 3, eps), err_msg=f"window {s}")
        np.testing.assert_array_equal(p2, oracle.perturb2(p1, dtype, g, seed, step, 3, -2 * eps, 4, eps),
                                      err_msg=f"window {s}")
        np.testing.assert_array_equal(p3, oracle.perturb2(p2, dtype, g, seed, step, 4, eps, 12, eps),
                                      err_msg=f"window {s}")
        want_u = oracle.update(p3, dtype, g, seed, step, c, lr)
        want_ur = oracle.update_restore(u, dtype, g, seed, step, c, lr, kr, eps)
        if dtype == "bf16":
            assert_bf16_within_1ulp(u, want_u, p3, c, lr)
        else:
            assert_f32_update_close(u, want_u, c, lr)
        assert_restore_update_close(ur, want_ur, u, c, lr, eps, dtype)


def test_full_size_separate_tensors():
    """OPT-13B as 644 separately allocated tensors, in the benchmark's per-tensor launch
    configuration (batches of 64 tensors per launch): a segmented perturb, two-probe transition,
    update and update-with-restore, checked against the oracle with each tensor's global offset
    on the first and last 2^15 weights of the first, last, largest and 24 random tensors."""
    w = workloads.WORKLOADS["opt13b"]
    spans = workloads.tensor_offsets(w)
    note(f"full-size opt13b as {len(spans)} tensors")
    tensors = [torch.empty(sz, dtype=torch.bfloat16, device=DEV) for _, _, sz in spans]
    offs = [o for _, o, _ in spans]
    workloads.fill_model_tensors_device(tensors, w)
    rng = np.random.default_rng(11)
    pick = {0, len(spans) - 1, int(np.argmax([sz for _, _, sz in spans]))}
    pick |= {int(i) for i in rng.integers(0, len(spans), 24)}
    part = 1 << 15
    wins = []  # (tensor index, local start, global start, length)
    for i in sorted(pick):
        sz = spans[i][2]
        for lo in sorted({0, max(sz - part, 0)}):
            wins.append((i, lo, offs[i] + lo, min(part, sz - lo)))
    grab = lambda: [host_bits(tensors[i][lo:lo + m]) for i, lo, _, m in wins]
    seed, step, K = 2024, 5, 16
    lp, lm, l0 = workloads.synthetic_losses(K, step)
    c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
    before = grab()
    zo.zo_perturb_segments(tensors, offs, 3, w.eps, 0, 0.0, seed, step)
    mid = grab()
    zo.zo_perturb_segments(tensors, offs, 3, -2 * w.eps, 4, w.eps, seed, step)
    trans = grab()
    zo.zo_update_segments(tensors, offs, c, w.lr, seed, step)
    after = grab()
    zo.zo_update_segments(tensors, offs, c, w.lr, seed, step, 4, -w.eps)
    final = grab()
    torch.cuda.synchronize()
    del tensors
    torch.cuda.empty_cache()
    for (i, lo, g, m), b, md, tr, a, f in zip(wins, before, mid, trans, after, final):
        np.testing.assert_array_equal(md, oracle.perturb(b, "bf16", g, seed, step, 3, w.eps), err_msg=f"tensor {i}")
        np.testing.assert_array_equal(tr, oracle.perturb2(md, "bf16", g, seed, step, 3, -2 * w.eps, 4, w.eps),
                                      err_msg=f"tensor {i}")
        assert_bf16_within_1ulp(a, oracle.update(tr, "bf16", g, seed, step, c, w.lr), tr, c, w.lr)
        assert_restore_update_close(f, oracle.update_restore(a, "bf16", g, seed, step, c, w.lr, 4, -w.eps),
                                    a, c, w.lr, -w.eps, "bf16")
