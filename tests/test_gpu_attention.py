"""GPU parity: rocs_dca_attention against the oracle (explicit K/V broadcast)."""

import numpy as np
import pytest
import torch

from gpu_util import assert_close, dev_bf16, dev_f32, dev_i32, host
from oracle import ikbo
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import ops
from paper_2607_27744_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (candidate counts, history lengths): empty requests, empty histories,
# histories of 1, around the 64-key stage and of two and three stages,
# candidate counts around the 128-row tile and its multiples.
SHAPES = [
    ([300, 1, 0, 211], [70, 5, 0, 129]),
    ([256, 257, 255], [64, 65, 63]),
    ([127, 128, 129], [128, 130, 191]),
    ([1], [1]),
    ([40, 500], [1000, 300]),
]


def _attn(case, scale=None):
    return host(ops.dca_attention(dev_bf16(case.q), dev_bf16(case.k), dev_bf16(case.v),
                                  dev_i32(case.cand_offsets), dev_i32(case.kv_offsets),
                                  scale=scale))


def _want(case, scale=None):
    return round_bf16(ikbo.dca_attention(case.q, case.k, case.v, case.cand_offsets,
                                         case.kv_offsets, scale=scale, mode="explicit"))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"n{sum(s[0])}-L{sum(s[1])}")
@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("q_len", [1, 3, 32, 64])
def test_attention_parity(gpu_lib, shape, head_dim, q_len):
    counts, lens = shape
    case = wl.attention_case(counts, lens, 2, head_dim, q_len=q_len, seed=head_dim + q_len)
    assert_close(_attn(case), _want(case), f"dca {shape} d{head_dim} T{q_len}")


def test_peaked_scores_exercise_rescaling(gpu_lib):
    # Large logits: the running max moves by far more than the lazy threshold.
    case = wl.attention_case([300, 90], [400, 257], 4, 64, seed=9, q_std=6.0)
    assert_close(_attn(case), _want(case), "peaked")
    assert_close(_attn(case, scale=0.01), _want(case, scale=0.01), "explicit scale")


@pytest.mark.parametrize("head_dim", [64, 128])
def test_running_max_jumps_past_the_weight_bound(gpu_lib, head_dim):
    # Scores far apart in the exp2 domain (more than 64 between stages), so
    # stages after the first must move the running max and redo their weights.
    case = wl.attention_case([300, 70], [700, 129], 2, head_dim, seed=11)
    assert_close(_attn(case, scale=4.0), _want(case, scale=4.0), f"scale 4 d{head_dim}")
    # A ramp: score of history row j is 64 (j mod 256) / 8 / sqrt(d), rising
    # by more than 64 (exp2 domain) from one 64-key stage to the next.
    q = np.zeros_like(case.q)
    q[..., 0] = 64.0
    k = np.zeros_like(case.k)
    local = np.concatenate([np.arange(n) for n in np.diff(case.kv_offsets)])
    k[:, :, 0] = ((local % 256) / 8.0)[:, None]
    ramp = type(case)(**{**vars(case), "q": q, "k": k})
    assert_close(_attn(ramp), _want(ramp), f"ramp d{head_dim}")


def test_single_key_is_exact(gpu_lib):
    # L = 1: the one weight is exactly 1, so the output is that value row.
    case = wl.attention_case([37, 300], [1, 1], 2, 128, seed=10, q_std=4.0)
    got = _attn(case)
    np.testing.assert_array_equal(got[:37, 0], np.broadcast_to(case.v[0], (37, 2, 128)))
    np.testing.assert_array_equal(got[37:, 0], np.broadcast_to(case.v[1], (300, 2, 128)))


def test_request_separation_probe(gpu_lib):
    # V rows of request r all equal 4 r: a candidate routed to the wrong
    # request would be off by at least 4.
    counts, lens = np.array([50, 0, 300, 7]), np.array([100, 64, 3, 190])
    case = wl.attention_case(counts, lens, 2, 64, seed=11)
    case.v = np.repeat(4.0 * np.repeat(np.arange(4), lens), 2 * 64).reshape(-1, 2, 64).astype(np.float32)
    got = _attn(case)
    want = np.repeat(4.0 * np.arange(4), counts)
    np.testing.assert_allclose(got, np.broadcast_to(want[:, None, None, None], got.shape), atol=0.02)


def test_strided_kv_slices_of_one_projection(gpu_lib):
    case = wl.attention_case([120, 130], [100, 140], 2, 64, seed=12)
    kv = torch.cat([dev_bf16(case.k).reshape(-1, 128), dev_bf16(case.v).reshape(-1, 128)], dim=1)
    k = kv[:, :128].view(-1, 2, 64)
    v = kv[:, 128:].view(-1, 2, 64)
    got = host(ops.dca_attention(dev_bf16(case.q), k, v, dev_i32(case.cand_offsets),
                                 dev_i32(case.kv_offsets)))
    assert_close(got, _want(case), "strided kv")


def test_general_path_fp32_and_small_head(gpu_lib):
    case = wl.attention_case([64, 64, 64, 64], [32, 32, 32, 32], 2, 32, seed=13, bf16=False)
    got = host(ops.dca_attention(dev_f32(case.q), dev_f32(case.k), dev_f32(case.v),
                                 dev_i32(case.cand_offsets), dev_i32(case.kv_offsets)))
    want = ikbo.dca_attention(case.q, case.k, case.v, case.cand_offsets, case.kv_offsets)
    assert_close(got, want, "fp32 d32", atol=1e-4, rtol=1e-4, normwise=1e-5)
    c16 = wl.attention_case([10, 0, 33], [7, 9, 0], 3, 40, seed=14)     # d = 40: general bf16
    assert_close(_attn(c16), _want(c16), "bf16 d40")


def test_deterministic_and_candidate_isolation(gpu_lib):
    case = wl.attention_case([500, 20], [300, 77], 2, 128, seed=15)
    a = _attn(case)
    np.testing.assert_array_equal(a, _attn(case))
    case.q = case.q.copy()
    case.q[7] = -case.q[7]
    b = _attn(case)
    keep = np.arange(a.shape[0]) != 7
    np.testing.assert_array_equal(a[keep], b[keep])


def test_mapped_attention_parity(gpu_lib):
    # rocs_dca_attention_mapped: candidates shuffled so each request's are
    # scattered; an empty history and a 1-key history included.
    for head_dim, bf16 in ((128, True), (64, True), (64, False)):
        case = wl.attention_case([37, 0, 90, 5, 21], [70, 5, 0, 129, 1], 2, head_dim, q_len=2,
                                 seed=40 + head_dim, bf16=bf16)
        perm = np.random.default_rng(head_dim).permutation(case.q.shape[0])
        q = np.ascontiguousarray(case.q[perm])
        m = ikbo.request_ids(case.cand_offsets)[perm]
        dev = dev_bf16 if bf16 else dev_f32
        got = host(ops.dca_attention_mapped(dev(q), dev(case.k), dev(case.v), dev_i32(m),
                                            dev_i32(case.kv_offsets)))
        want = ikbo.dca_attention(q, case.k, case.v, None, case.kv_offsets, request_map=m)
        assert_close(got, round_bf16(want) if bf16 else want, f"mapped d{head_dim} bf16={bf16}")


@pytest.mark.parametrize("head_dim,bf16", [(128, True), (64, True), (64, False)],
                         ids=["d128-bf16", "d64-bf16", "d64-fp32"])
def test_mapped_attention_index_probe_bit_exact(gpu_lib, head_dim, bf16):
    # Every request has a history of one row whose values are all 4 r, so the
    # one softmax weight is exactly 1 and candidate n's output is exactly
    # 4 m_n: the device's handling of a shuffled per-candidate map is checked
    # bit for bit (a wrong request is off by at least 4).
    n_req = 37
    counts = np.random.default_rng(head_dim).integers(0, 60, size=n_req)
    counts[[3, 20]] = 0
    case = wl.attention_case(counts, np.ones(n_req, np.int64), 2, head_dim, q_len=2,
                             seed=60 + head_dim, bf16=bf16, q_std=3.0)
    case.v = np.broadcast_to(4.0 * np.arange(n_req, dtype=np.float32)[:, None, None],
                             case.v.shape).copy()
    perm = np.random.default_rng(7).permutation(case.q.shape[0])
    m = ikbo.request_ids(case.cand_offsets)[perm]
    dev = dev_bf16 if bf16 else dev_f32
    got = host(ops.dca_attention_mapped(dev(np.ascontiguousarray(case.q[perm])), dev(case.k),
                                        dev(case.v), dev_i32(m), dev_i32(case.kv_offsets)))
    want = np.broadcast_to((4.0 * m)[:, None, None, None], got.shape)
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("head_dim", [64, 128])
def test_mapped_grouping_and_tiled_parity(gpu_lib, head_dim):
    # The mapped form groups the candidates by request on the device (a
    # stable counting sort over blocks of 4096 candidates) and runs the tiled
    # kernel in grouped order. The grouping left in the workspace must be
    # NumPy's stable argsort of the map and the offsets of its counts, bit
    # for bit; the outputs match the oracle. About 14k candidates (four
    # grouping blocks), 41 requests of which three are empty, one with a
    # single candidate, histories of 1 .. 300 rows, two query tokens.
    rng = np.random.default_rng(head_dim)
    counts = rng.integers(150, 600, size=41)
    counts[[4, 17, 30]] = 0
    counts[9] = 1
    lens = rng.integers(1, 300, size=41)
    case = wl.attention_case(counts, lens, 2, head_dim, q_len=2, seed=80 + head_dim)
    n = case.q.shape[0]
    perm = rng.permutation(n)
    m = ikbo.request_ids(case.cand_offsets)[perm].astype(np.int32)
    q = np.ascontiguousarray(case.q[perm])
    ws = torch.zeros(ops.dca_attention_mapped_workspace_size(41, n), dtype=torch.uint8,
                     device="cuda")
    got = host(ops.dca_attention_mapped(dev_bf16(q), dev_bf16(case.k), dev_bf16(case.v),
                                        dev_i32(m), dev_i32(case.kv_offsets), workspace=ws))
    want = ikbo.dca_attention(q, case.k, case.v, None, case.kv_offsets, request_map=m)
    assert_close(got, round_bf16(want), f"mapped tiled d{head_dim}")
    raw = ws.cpu().numpy().view(np.int32)
    grp_off = raw[:42]
    order = raw[256 // 4 * ((42 * 4 + 255) // 256):][:n]
    np.testing.assert_array_equal(order, np.argsort(m, kind="stable"))
    np.testing.assert_array_equal(grp_off, np.concatenate([[0], np.cumsum(np.bincount(m, minlength=41))]))
    # Every row equals the CSR kernel's row for the same candidate: grouping
    # only reorders which rows share a tile.
    csr = host(ops.dca_attention(dev_bf16(case.q), dev_bf16(case.k), dev_bf16(case.v),
                                 dev_i32(case.cand_offsets), dev_i32(case.kv_offsets)))
    np.testing.assert_array_equal(got, csr[perm])


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("q_len", [1, 32])
def test_request_side_attention(gpu_lib, head_dim, q_len):
    # A^R = Attn(Q^R, K, V): each request's own queries over its history
    # (Eq. dca-attention), run as the identity map on the tiled kernel.
    lens = [300, 0, 64, 1, 1000]
    case = wl.attention_case([1] * len(lens), lens, 4, head_dim, q_len=q_len, seed=50 + q_len)
    got = host(ops.dca_request_attention(dev_bf16(case.q), dev_bf16(case.k), dev_bf16(case.v),
                                         dev_i32(case.kv_offsets)))
    want = ikbo.dca_attention(case.q, case.k, case.v, np.arange(len(lens) + 1),
                              case.kv_offsets)
    assert_close(got, round_bf16(want), f"request-side d{head_dim} T{q_len}")


@pytest.mark.parametrize("shape", SHAPES[:3] + [([5, 40], [0, 70])],
                         ids=lambda s: f"n{sum(s[0])}-L{sum(s[1])}")
@pytest.mark.parametrize("head_dim", [64, 128])
def test_attention_residual(gpu_lib, shape, head_dim):
    # The stacked-DCA residual formed in the epilogue: out is exactly the
    # plain call's output, out_sum = round(out + residual) in fp32 (RNE), and
    # an empty history passes the residual through.
    counts, lens = shape
    case = wl.attention_case(counts, lens, 2, head_dim, seed=head_dim + 5)
    rng = np.random.default_rng(head_dim)
    res = round_bf16(rng.standard_normal(case.q.shape))
    args = (dev_bf16(case.q), dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    plain = ops.dca_attention(*args)
    out, out_sum = ops.dca_attention_residual(*args, dev_bf16(res))
    torch.cuda.synchronize()
    assert torch.equal(out, plain)
    want_sum = (out.float() + dev_bf16(res).float()).to(torch.bfloat16)
    assert torch.equal(out_sum, want_sum)
    # Against the oracle: u = round(round(A) + residual).
    want = round_bf16(ikbo.dca_attention(case.q, case.k, case.v, case.cand_offsets,
                                         case.kv_offsets))
    assert_close(host(out_sum), round_bf16(want + res), f"residual {shape} d{head_dim}")


def test_attention_residual_general_kernel_fp32(gpu_lib):
    # fp32 runs the general kernel: out_sum = out + residual exactly.
    case = wl.attention_case([33, 0, 70], [20, 9, 0], 2, 32, seed=3, bf16=False)
    res = np.random.default_rng(1).standard_normal(case.q.shape)
    args = (dev_f32(case.q), dev_f32(case.k), dev_f32(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    out, out_sum = ops.dca_attention_residual(*args, dev_f32(res))
    torch.cuda.synchronize()
    assert torch.equal(out_sum, out + dev_f32(res))
    want = ikbo.dca_attention(case.q, case.k, case.v, case.cand_offsets, case.kv_offsets)
    assert_close(host(out), want, "fp32 attention", atol=1e-4, rtol=1e-4)


def _proj_case(counts, lens, heads, dim, d_in, seed, bf16=True, q_len=1):
    case = wl.attention_case(counts, lens, heads, dim, seed=seed, bf16=bf16, q_len=q_len)
    rnd = round_bf16 if bf16 else (lambda a: a)
    x = wl.normal(wl.tensor_rng(seed, 210, 1), (case.n_cand, q_len, d_in), bf16=bf16)
    wq = wl.normal(wl.tensor_rng(seed, 210, 2), (heads * dim, d_in), std=d_in ** -0.5, bf16=bf16)
    res = wl.normal(wl.tensor_rng(seed, 210, 3), (case.n_cand, q_len, heads, dim), bf16=bf16)
    q = ikbo.linear(x.reshape(-1, d_in), wq).reshape(case.n_cand, q_len, heads, dim)
    want = ikbo.dca_attention(rnd(q), case.k, case.v, case.cand_offsets, case.kv_offsets)
    return case, x, wq, res, rnd(want)


@pytest.mark.parametrize("shape,q_len", [(s, 1) for s in SHAPES[:4]] +
                         [(([5, 40], [0, 70]), 1), (SHAPES[0], 3)],
                         ids=lambda s: f"n{sum(s[0])}-L{sum(s[1])}" if isinstance(s, tuple) else f"T{s}")
def test_attention_proj_matches_project_then_attend(gpu_lib, shape, q_len):
    # The fused query projection (head_dim 64, d_in 256) uses the streaming
    # linear's operand roles and k order: out and out_sum equal projecting
    # with rocs_ikbo_linear and then attending, bit for bit.
    counts, lens = shape
    case, x, wq, res, want = _proj_case(counts, lens, 4, 64, 256, seed=21, q_len=q_len)
    X, WQ, RES = dev_bf16(x), dev_bf16(wq), dev_bf16(res)
    args = (dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    q = ops.ikbo_linear(X.view(-1, 256), WQ).view(-1, q_len, 4, 64)
    ref_out, ref_sum = ops.dca_attention_residual(q, *args, RES)
    out, out_sum = ops.dca_attention_proj(X, WQ, *args, heads=4, residual=RES)
    plain = ops.dca_attention_proj(X, WQ, *args, heads=4)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out)
    assert torch.equal(out_sum, ref_sum)
    assert torch.equal(plain, ref_out)
    assert_close(host(out), want, f"proj {shape}")


@pytest.mark.parametrize("dim,d_in,bf16", [(128, 256, True), (64, 96, True), (32, 48, False)])
def test_attention_proj_general_kernel(gpu_lib, dim, d_in, bf16):
    case, x, wq, res, want = _proj_case([33, 0, 70], [20, 9, 100], 2, dim, d_in, seed=dim,
                                        bf16=bf16)
    dev = dev_bf16 if bf16 else dev_f32
    args = (dev(case.k), dev(case.v), dev_i32(case.cand_offsets), dev_i32(case.kv_offsets))
    out, out_sum = ops.dca_attention_proj(dev(x), dev(wq), *args, heads=2, residual=dev(res))
    torch.cuda.synchronize()
    tol = {} if bf16 else dict(atol=1e-4, rtol=1e-4)
    assert_close(host(out), want, f"proj general d{dim} in{d_in}", **tol)
    want_sum = (out.float() + dev(res).float()).to(out.dtype)
    assert torch.equal(out_sum, want_sum)


def _plan_want(co, ko, heads, q_len=1, rows=128):
    """The tile plan the kernel order follows, from its definition: requests by
    history length, longest first (lengths from 2^20 - 1 on count as equal;
    ties by index), and the running sum of heads * ceil(n_r q_len / rows) in
    that order."""
    co, ko = np.asarray(co, np.int64), np.asarray(ko, np.int64)
    lens = np.minimum(np.diff(ko), (1 << 20) - 1)
    order = sorted(range(lens.size), key=lambda r: (-lens[r], r))
    tiles = [heads * -(-(int(co[r + 1] - co[r]) * q_len) // rows) for r in order]
    return np.array(order, np.int64), np.concatenate([[0], np.cumsum(tiles)]).astype(np.int64)


def _many(r, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 300, r).tolist(), rng.integers(0, 2000, r).tolist()


@pytest.mark.parametrize("counts,lens", [
    ([300, 1, 0, 211], [70, 5, 0, 129]),
    ([5, 7, 9, 11, 13], [64, 64, 300, 64, 300]),          # ties keep index order
    ([1], [1]),
    ([40, 0, 7], [0, 0, 0]),                              # every history empty
    ([], []),                                             # no requests
    _many(256, 1),                                        # largest counted ranking
    _many(257, 2),                                        # smallest bitonic sort
    (list(range(0, 3000, 3)), [(37 * r) % 1500 for r in range(1000)]),
    _many(4096, 3),                                       # largest sorted plan
], ids=["ragged", "ties", "one", "empty-histories", "none", "r256", "r257", "r1000", "r4096"])
@pytest.mark.parametrize("heads,q_len", [(4, 1), (2, 3)])
def test_attention_plan_contents(gpu_lib, counts, lens, heads, q_len):
    co = wl.offsets_from_counts(np.asarray(counts))
    ko = wl.offsets_from_counts(np.asarray(lens))
    plan = ops.dca_attention_plan(dev_i32(co), dev_i32(ko), num_cand=int(co[-1]), heads=heads,
                                  q_len=q_len)
    torch.cuda.synchronize()
    got = plan.view(torch.int32).cpu().numpy().astype(np.int64)
    r = len(counts)
    order, pref = _plan_want(co, ko, heads, q_len)
    assert got[0] == 1 and got[1] == pref[-1] and got[2] == r and got[3] == heads
    assert got[4] == q_len and got[5] == 128
    np.testing.assert_array_equal(got[8:8 + r], order)
    np.testing.assert_array_equal(got[8 + r:8 + 2 * r + 1], pref)


def test_attention_plan_beyond_the_sort_keeps_the_builtin_order(gpu_lib):
    # 5000 requests: the plan records mode 0 and the kernel's own order runs.
    rng = np.random.default_rng(5)
    counts, lens = rng.integers(0, 40, 5000), rng.integers(0, 90, 5000)
    case = wl.attention_case(counts, lens, 2, 64, seed=3)
    args = (dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    plan = ops.dca_attention_plan(args[2], args[3], num_cand=case.n_cand, heads=2)
    torch.cuda.synchronize()
    head = plan.view(torch.int32)[:8].cpu().numpy()
    assert head[0] == 0 and head[2] == 5000
    q = dev_bf16(case.q)
    torch.testing.assert_close(ops.dca_attention_ex(q, *args, plan=plan),
                               ops.dca_attention(q, *args), rtol=0, atol=0)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"n{sum(s[0])}-L{sum(s[1])}")
@pytest.mark.parametrize("head_dim,q_len", [(64, 1), (128, 1), (64, 3)])
def test_attention_with_plan_is_bit_identical(gpu_lib, shape, head_dim, q_len):
    # The plan only reorders whole tiles: every output bit is the same, and a
    # plan made for other heads or q_len is ignored.
    counts, lens = shape
    case = wl.attention_case(counts, lens, 2, head_dim, q_len=q_len, seed=7)
    q = dev_bf16(case.q)
    args = (dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    ref = ops.dca_attention(q, *args)
    plan = ops.dca_attention_plan(args[2], args[3], num_cand=case.n_cand, heads=2, q_len=q_len)
    other = ops.dca_attention_plan(args[2], args[3], num_cand=case.n_cand, heads=3, q_len=q_len)
    got = ops.dca_attention_ex(q, *args, plan=plan)
    got_other = ops.dca_attention_ex(q, *args, plan=other)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    assert torch.equal(got_other, ref)
    assert_close(host(got), _want(case), f"planned {shape} d{head_dim} T{q_len}")


@pytest.mark.parametrize("q_len", [1, 3])
def test_attention_ex_all_options(gpu_lib, q_len):
    # Projection, residual and plan together, several query tokens: equal to
    # the three-call composition (project, attend, add) bit for bit.
    case, x, wq, res, want = _proj_case([129, 0, 300, 1, 64], [700, 9, 0, 64, 1], 4, 64, 256,
                                        seed=31, q_len=q_len)
    X, WQ, RES = dev_bf16(x), dev_bf16(wq), dev_bf16(res)
    args = (dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    plan = ops.dca_attention_plan(args[2], args[3], num_cand=case.n_cand, heads=4, q_len=q_len)
    out, out_sum = ops.dca_attention_ex(X, *args, w_q=WQ, heads=4, plan=plan, residual=RES)
    q = ops.ikbo_linear(X.view(-1, 256), WQ).view(-1, q_len, 4, 64)
    ref = ops.dca_attention(q, *args)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    assert torch.equal(out_sum, (ref.float() + RES.float()).to(torch.bfloat16))
    assert_close(host(out), want, f"ex T{q_len}")


def test_attention_proj_with_plan(gpu_lib):
    case, x, wq, res, want = _proj_case([300, 1, 0, 211, 40], [70, 5, 0, 129, 1000], 4, 64, 256,
                                        seed=23)
    X, WQ, RES = dev_bf16(x), dev_bf16(wq), dev_bf16(res)
    args = (dev_bf16(case.k), dev_bf16(case.v), dev_i32(case.cand_offsets),
            dev_i32(case.kv_offsets))
    plan = ops.dca_attention_plan(args[2], args[3], num_cand=case.n_cand, heads=4)
    ref_out, ref_sum = ops.dca_attention_proj(X, WQ, *args, heads=4, residual=RES)
    out, out_sum = ops.dca_attention_proj(X, WQ, *args, heads=4, residual=RES, plan=plan)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(out_sum, ref_sum)
    assert_close(host(out), want, "proj planned")
