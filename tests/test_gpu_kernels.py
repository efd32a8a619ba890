"""Per-kernel parity: every HIP kernel of the block against the oracle step
it computes (or, for a bare GEMM, its plain definition), through the
test-only C entry points.  Sizes span several tiles plus a ragged tail."""

import math

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import DTYPES, TOL, dev, dev_i32, host, rel_l2, rnd, sync

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2406_14898_amd import flglm as F  # noqa: E402

DT = ["bf16", "f32"]


# ---------------------------------------------------------------------------
# GEMM: three layouts, every epilogue
# ---------------------------------------------------------------------------

def _gelu(z):
    return oracle.gelu(z)


@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("epi", [F.FL_EPI_STORE, F.FL_EPI_BIAS, F.FL_EPI_BIAS_RES, F.FL_EPI_BIAS_GELU])
@pytest.mark.parametrize("N", [512, 384])
@pytest.mark.parametrize("M", [300, 400])
def test_gemm_nt(dt, epi, N, M):
    """M = 300 / 400: the last 256-row tile ends inside its first / second
    128-row epilogue half."""
    code, tdt = DTYPES[dt]
    K = 320
    A, B = rnd((M, K), 1, dt=dt), rnd((N, K), 2, 0.1, dt=dt)
    bias, R = rnd((N,), 3, dt=dt), rnd((M, N), 4, dt=dt)
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    if epi != F.FL_EPI_STORE:
        ref = ref + bias
    if epi == F.FL_EPI_BIAS_RES:
        ref = ref + R
    dA, dB, dbias, dR = dev(A, dt), dev(B, dt), dev(bias, dt), dev(R, dt)
    C = torch.full((M, N), float("nan"), dtype=tdt, device="cuda")
    C2 = torch.full((M, N), float("nan"), dtype=tdt, device="cuda")
    F.fl_test_gemm(code, F.FL_GEMM_NT, epi, dA, dB, C, M, N, K, K, K, N, bias=dbias, R=dR, ldr=N, C2=C2, ldc2=N)
    sync()
    assert rel_l2(host(C), ref) < TOL[dt] / 4
    if epi == F.FL_EPI_BIAS_GELU:
        assert rel_l2(host(C2), _gelu(ref)) < TOL[dt] / 4


@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("epi", [F.FL_EPI_STORE, F.FL_EPI_GELU_BWD])
@pytest.mark.parametrize("N", [384, 512])
def test_gemm_nn(dt, epi, N):
    code, tdt = DTYPES[dt]
    M, K = 420, 448
    A, B, Z = rnd((M, K), 5, dt=dt), rnd((K, N), 6, 0.1, dt=dt), rnd((M, N), 7, dt=dt)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    if epi == F.FL_EPI_GELU_BWD:
        ref = ref * oracle.gelu_grad(Z.astype(np.float64))
    C = torch.full((M, N), float("nan"), dtype=tdt, device="cuda")
    F.fl_test_gemm(code, F.FL_GEMM_NN, epi, dev(A, dt), dev(B, dt), C, M, N, K, K, N, N, Z=dev(Z, dt), ldz=N)
    sync()
    assert rel_l2(host(C), ref) < TOL[dt] / 4


@pytest.mark.parametrize("M", [700, 256, 1])
def test_gemm_gelu_bwd_column_sums(M):
    """The GeLU' input-gradient GEMM also writes, per 256-row block, the
    column sums of what it stores (the bias gradient's partial sums): equal
    to the sums of the stored bf16 values over each block's rows, up to fp32
    summation order.  M = 700 ends a block inside its second 128-row half."""
    N, K = 768, 448
    A, B, Z = rnd((M, K), 21, dt="bf16"), rnd((K, N), 22, 0.1, dt="bf16"), rnd((M, N), 23, dt="bf16")
    C = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    nb = (M + 255) // 256
    cs = torch.full((nb, N), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_NN, F.FL_EPI_GELU_BWD, dev(A, "bf16"), dev(B, "bf16"), C, M, N, K, K, N, N,
                   Z=dev(Z, "bf16"), ldz=N, colsum=cs)
    sync()
    c = host(C).astype(np.float64)
    ref = A.astype(np.float64) @ B.astype(np.float64) * oracle.gelu_grad(Z.astype(np.float64))
    assert rel_l2(c, ref) < TOL["bf16"] / 4
    got = host(cs)
    for b in range(nb):
        want = c[256 * b:256 * (b + 1)].sum(axis=0)
        scale = np.abs(c[256 * b:256 * (b + 1)]).sum(axis=0) + 1e-30
        assert np.all(np.abs(got[b] - want) <= 1e-6 * scale), b


def test_gemm_column_sums_only_where_supported():
    """Column sums come only from the bf16 GeLU' input-gradient GEMM on the
    LDS-DMA kernel; elsewhere the call is refused before any work."""
    M, N, K = 300, 512, 256
    cs = torch.zeros((2, N), dtype=torch.float32, device="cuda")
    for dt, lay, epi, n in (("f32", F.FL_GEMM_NN, F.FL_EPI_GELU_BWD, N), ("bf16", F.FL_GEMM_NN, F.FL_EPI_STORE, N),
                            ("bf16", F.FL_GEMM_NN, F.FL_EPI_GELU_BWD, 384)):
        code, tdt = DTYPES[dt]
        A = torch.zeros((M, K), dtype=tdt, device="cuda")
        B = torch.zeros((K, n), dtype=tdt, device="cuda")
        C = torch.zeros((M, n), dtype=tdt, device="cuda")
        with pytest.raises(F.FlglmError) as e:
            F.fl_test_gemm(code, lay, epi, A, B, C, M, n, K, K, n, n, Z=C, ldz=n, colsum=cs)
        assert e.value.code == F.FL_ERR_ARG


@pytest.mark.parametrize("dt", DT)
def test_gemm_tn_accumulates(dt):
    code, tdt = DTYPES[dt]
    M, N, K = 272, 512, 300  # K (tokens) ragged
    A, B = rnd((K, M), 8, dt=dt), rnd((K, N), 9, dt=dt)
    C0 = rnd((M, N), 10, dt="f32")
    ref = C0.astype(np.float64) + A.astype(np.float64).T @ B.astype(np.float64)
    C = torch.from_numpy(C0).cuda()
    F.fl_test_gemm(code, F.FL_GEMM_TN, F.FL_EPI_ACC_F32, dev(A, dt), dev(B, dt), C, M, N, K, M, N, N)
    sync()
    assert rel_l2(host(C), ref) < (1e-5 if dt == "f32" else 5e-3)


@pytest.mark.parametrize("K", [1, 63, 64, 65, 128, 129, 192])
def test_gemm_tn_short_reductions(K):
    """bf16 weight gradient over 1-3 reduction stages: the prologue and peeled
    last stage of the loop, where only some waves issue the operand loads."""
    M, N = 256, 512
    A, B = rnd((K, M), 60 + K), rnd((K, N), 61 + K)
    C0 = rnd((M, N), 62, dt="f32")
    ref = C0.astype(np.float64) + A.astype(np.float64).T @ B.astype(np.float64)
    C = torch.from_numpy(C0).cuda()
    F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_TN, F.FL_EPI_ACC_F32, dev(A, "bf16"), dev(B, "bf16"), C, M, N, K, M, N, N)
    sync()
    assert rel_l2(host(C), ref) < 5e-3


SPLIT_CASES = [  # (layout, epi, M, N, K): 1-4 tiles, K of 128+ stages, so the launch splits the reduction
    (F.FL_GEMM_NT, F.FL_EPI_BIAS_RES, 300, 512, 8192),
    (F.FL_GEMM_NT, F.FL_EPI_BIAS_GELU, 200, 256, 8256),
    (F.FL_GEMM_NN, F.FL_EPI_STORE, 420, 256, 8192),
    (F.FL_GEMM_NN, F.FL_EPI_GELU_BWD, 300, 512, 8192),
    (F.FL_GEMM_TN, F.FL_EPI_ACC_F32, 272, 512, 8300),
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: f"L{c[0]}E{c[1]}M{c[2]}N{c[3]}K{c[4]}")
def test_gemm_split_reduction(case):
    """bf16: the partial last round of tiles split into reduction slices (fp32
    partials in scratch, fixed-order fixup) against fp64 and the unsplit run."""
    lay, epi, M, N, K = case
    rng = 40 + epi
    if lay == F.FL_GEMM_NT:
        A, B, lda, ldb = rnd((M, K), rng), rnd((N, K), rng + 1, 0.05), K, K
        ref = A.astype(np.float64) @ B.astype(np.float64).T
    elif lay == F.FL_GEMM_NN:
        A, B, lda, ldb = rnd((M, K), rng), rnd((K, N), rng + 1, 0.05), K, N
        ref = A.astype(np.float64) @ B.astype(np.float64)
    else:
        A, B, lda, ldb = rnd((K, M), rng), rnd((K, N), rng + 1), M, N
        ref = A.astype(np.float64).T @ B.astype(np.float64)
    bias, R, Z = rnd((N,), rng + 2), rnd((M, N), rng + 3), rnd((M, N), rng + 4)
    C0 = rnd((M, N), rng + 5, dt="f32")
    if epi in (F.FL_EPI_BIAS_RES, F.FL_EPI_BIAS_GELU):
        ref = ref + bias
    if epi == F.FL_EPI_BIAS_RES:
        ref = ref + R
    if epi == F.FL_EPI_GELU_BWD:
        ref = ref * oracle.gelu_grad(Z.astype(np.float64))
    if epi == F.FL_EPI_ACC_F32:
        ref = ref + C0
    outs = []
    for part in (None, torch.zeros(64 << 20 >> 2, dtype=torch.float32, device="cuda")):
        if epi == F.FL_EPI_ACC_F32:
            C = torch.from_numpy(C0.copy()).cuda()
        else:
            C = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        C2 = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        F.fl_test_gemm(F.FL_BF16, lay, epi, dev(A, "bf16"), dev(B, "bf16"), C, M, N, K, lda, ldb, N,
                       bias=dev(bias, "bf16"), R=dev(R, "bf16"), ldr=N, C2=C2, ldc2=N, Z=dev(Z, "bf16"), ldz=N,
                       part=part)
        sync()
        outs.append((host(C), host(C2)))
        tol = 5e-3 if epi == F.FL_EPI_ACC_F32 else TOL["bf16"] / 4
        assert rel_l2(outs[-1][0], ref) < tol
        if epi == F.FL_EPI_BIAS_GELU:
            assert rel_l2(outs[-1][1], _gelu(ref)) < TOL["bf16"] / 4
    # the split run differs from the unsplit one only by fp32 summation order
    assert rel_l2(outs[1][0], outs[0][0]) < 1e-2


def test_gemm_rejects_bad_shapes():
    A = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(F.FlglmError):
        F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_NT, F.FL_EPI_STORE, A, A, A, 64, 100, 64, 64, 64, 100)
    with pytest.raises(F.FlglmError):  # K not a multiple of 64 with a K-contiguous operand
        F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_NT, F.FL_EPI_STORE, A, A, A, 64, 128, 40, 64, 64, 128)
    with pytest.raises(F.FlglmError):  # unsupported layout / epilogue pair
        F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_TN, F.FL_EPI_BIAS, A, A, A, 64, 128, 64, 64, 128, 128)


# ---------------------------------------------------------------------------
# LayerNorm and column sums
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("H", [256, 4096])
def test_layernorm_fwd_bwd(dt, H):
    code, tdt = DTYPES[dt]
    T = 37
    x = rnd((T, H), 11, 2.0, dt=dt) + np.float32(0.5)
    x = synth.bf16_round(x) if dt == "bf16" else x
    g = rnd((H,), 12, 0.1, dt=dt) + np.float32(1.0)
    g = synth.bf16_round(g) if dt == "bf16" else g
    b = rnd((H,), 13, 0.1, dt=dt)
    y_ref, xhat, rstd = oracle.layer_norm(x.astype(np.float64), g, b, 1e-5)
    dx_, dg_, db_ = dev(x, dt), dev(g, dt), dev(b, dt)
    y = torch.empty((T, H), dtype=tdt, device="cuda")
    mean = torch.empty(T, dtype=torch.float32, device="cuda")
    rs = torch.empty(T, dtype=torch.float32, device="cuda")
    F.fl_test_layernorm_fwd(code, dx_, dg_, db_, y, mean, rs, T, H, 1e-5)
    sync()
    assert rel_l2(host(y), y_ref) < TOL[dt] / 4
    assert rel_l2(host(rs), rstd[:, 0]) < 1e-5
    assert rel_l2(host(mean), x.astype(np.float64).mean(1)) < 1e-5

    dy = rnd((T, H), 14, dt=dt)
    dres = rnd((T, H), 15, dt=dt)
    dxr, dgr, dbr = oracle.layer_norm_backward(dy.astype(np.float64), xhat, rstd, g.astype(np.float64))
    out = torch.empty((T, H), dtype=tdt, device="cuda")
    F.fl_test_layernorm_bwd(code, dev(dy, dt), dx_, mean, rs, dg_, dev(dres, dt), out, T, H)
    sync()
    assert rel_l2(host(out), dxr + dres) < TOL[dt] / 4
    og = torch.zeros(H, dtype=torch.float32, device="cuda")
    ob = torch.ones(H, dtype=torch.float32, device="cuda")
    part = torch.empty(2 * H * ((T + 255) // 256), dtype=torch.float32, device="cuda")
    F.fl_test_colsum(code, 1, dev(dy, dt), dx_, mean, rs, T, H, og, ob, part)
    sync()
    assert rel_l2(host(og), dgr) < 1e-4
    assert rel_l2(host(ob), dbr + 1.0) < 1e-5


@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("H,T", [(256, 3), (768, 513), (4096, 2011)])
@pytest.mark.parametrize("with_res", [True, False])
def test_layernorm_bwd_fused(dt, H, T, with_res):
    """The stack's LayerNorm backward with its column sums in the same pass:
    dx (with and without the residual term), the gain and shift gradients and
    the column sums of dx, against the oracle's LayerNorm backward.  T = 3
    leaves most of the 512 row blocks empty; T = 2011 splits unevenly."""
    code, tdt = DTYPES[dt]
    x = rnd((T, H), 31, 2.0, dt=dt) + np.float32(0.5)
    x = synth.bf16_round(x) if dt == "bf16" else x
    g = rnd((H,), 32, 0.1, dt=dt) + np.float32(1.0)
    g = synth.bf16_round(g) if dt == "bf16" else g
    b = rnd((H,), 33, 0.1, dt=dt)
    _, xhat, rstd = oracle.layer_norm(x.astype(np.float64), g, b, 1e-5)
    dx_, dg_ = dev(x, dt), dev(g, dt)
    mean = torch.from_numpy(x.astype(np.float64).mean(1).astype(np.float32)).cuda()
    rs = torch.from_numpy(rstd[:, 0].astype(np.float32)).cuda()
    dy = rnd((T, H), 34, dt=dt)
    dres = rnd((T, H), 35, dt=dt) if with_res else np.zeros((T, H), np.float32)
    dxr, dgr, dbr = oracle.layer_norm_backward(dy.astype(np.float64), xhat, rstd, g.astype(np.float64))
    out = torch.full((T, H), float("nan"), dtype=tdt, device="cuda")
    og = torch.zeros(H, dtype=torch.float32, device="cuda")
    ob = torch.ones(H, dtype=torch.float32, device="cuda")
    osum = torch.full((H,), 2.0, dtype=torch.float32, device="cuda")
    part = torch.full((3 * 512 * H,), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_layernorm_bwd_fused(code, dev(dy, dt), dx_, mean, rs, dg_, dev(dres, dt) if with_res else None, out,
                                  T, H, og, ob, osum, part)
    sync()
    got = host(out)
    assert rel_l2(got, dxr + dres) < TOL[dt] / 4
    assert rel_l2(host(og), dgr) < 1e-4
    assert rel_l2(host(ob), dbr + 1.0) < 1e-5
    # the sum of what was stored (rounded), added in fp32
    assert rel_l2(host(osum), got.sum(0) + 2.0) < 1e-5
    # dx only: no sums asked for, no scratch needed
    out2 = torch.full((T, H), float("nan"), dtype=tdt, device="cuda")
    F.fl_test_layernorm_bwd_fused(code, dev(dy, dt), dx_, mean, rs, dg_, dev(dres, dt) if with_res else None, out2,
                                  T, H)
    sync()
    assert torch.equal(out2, out)


@pytest.mark.parametrize("dt", DT)
def test_colsum_many_blocks(dt):
    code, _ = DTYPES[dt]
    T, N = 1000, 1536
    X = rnd((T, N), 16, dt=dt)
    out = torch.zeros(N, dtype=torch.float32, device="cuda")
    part = torch.empty(2 * N * ((T + 255) // 256), dtype=torch.float32, device="cuda")
    F.fl_test_colsum(code, 0, dev(X, dt), None, None, None, T, N, out, None, part)
    F.fl_test_colsum(code, 0, dev(X, dt), None, None, None, T, N, out, None, part)
    sync()
    assert rel_l2(host(out), 2 * X.astype(np.float64).sum(0)) < 1e-5


# ---------------------------------------------------------------------------
# Rotary and attention
# ---------------------------------------------------------------------------

def _many_tiny():
    """600 sequences of 1 to 4 tokens, three per client: many (sequence, head)
    groups, every tile ragged."""
    lens = np.random.default_rng(9).integers(1, 5, 600)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return synth.Batch(cu, np.arange(0, 601, 3, dtype=np.int32))


BATCHES = {
    "ragged_causal": synth.Batch(np.array([0, 1, 6, 70, 135, 335], np.int32), np.array([0, 2, 5], np.int32)),
    "ragged_prefix": synth.Batch(np.array([0, 1, 6, 70, 135, 335], np.int32), np.array([0, 2, 5], np.int32),
                                 "prefix", np.array([0, 3, 16, 65, 150], np.int32)),
    # contexts covering the whole sequence (bidirectional) or all but its last token
    "full_context": synth.Batch(np.array([0, 1, 65, 130, 260], np.int32), np.array([0, 1, 4], np.int32),
                                "prefix", np.array([1, 64, 64, 130], np.int32)),
    "many_tiny": _many_tiny(),
}


def _qkv(T, H, seed, dt):
    return rnd((T, 3 * H), seed, dt=dt)


@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("heads", [(2, 128), (4, 64)])
def test_rope_inplace(dt, heads):
    code, tdt = DTYPES[dt]
    nh, d = heads
    H = nh * d
    r = d // 2
    b = BATCHES["ragged_causal"]
    T = b.total_tokens
    qkv = _qkv(T, H, 20, dt)
    t = dev(qkv, dt)
    pos = torch.empty(T, dtype=torch.int32, device="cuda")
    ct = torch.empty(b.max_seqlen * r // 2, dtype=torch.float32, device="cuda")
    st = torch.empty_like(ct)
    F.fl_test_rope(code, t, dev_i32(b.cu_seqlens), b.num_seqs, T, b.max_seqlen, H, nh, r, 10000.0, pos, ct, st)
    sync()
    p = oracle.positions(b.cu_seqlens)
    np.testing.assert_array_equal(pos.cpu().numpy(), p)
    cos, sin = oracle.rope_tables(p, r, 10000.0)
    out = host(t)
    q = oracle.rope(qkv[:, :H].astype(np.float64).reshape(T, nh, d), cos, sin, r).reshape(T, H)
    k = oracle.rope(qkv[:, H:2 * H].astype(np.float64).reshape(T, nh, d), cos, sin, r).reshape(T, H)
    assert rel_l2(out[:, :H], q) < TOL[dt] / 4
    assert rel_l2(out[:, H:2 * H], k) < TOL[dt] / 4
    np.testing.assert_array_equal(out[:, 2 * H:], qkv[:, 2 * H:])


def _lse_ref(q, k, b):
    T, nh, d = q.shape
    out = np.zeros((T, nh))
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        P = int(b.prefix_len[s]) if b.mask == "prefix" else None
        allowed = oracle.allowed_mask(r1 - r0, P)
        for h in range(nh):
            S = q[r0:r1, h] @ k[r0:r1, h].T / math.sqrt(d)
            S = np.where(allowed, S, -np.inf)
            m = S.max(1, keepdims=True)
            out[r0:r1, h] = (m + np.log(np.exp(S - m).sum(1, keepdims=True)))[:, 0]
    return out


def _ds_work(cu_seqlens, prefix_len, nh, num_prefix=0):
    """Device workspace for the stored softmax gradient of a bf16 backward."""
    n = F.fl_test_attention_ds_bytes(np.asarray(cu_seqlens), prefix_len, nh, num_prefix)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("dt", DT)
@pytest.mark.parametrize("heads", [(2, 128), (4, 64)])
@pytest.mark.parametrize("bname", list(BATCHES))
def test_attention_fwd_bwd(dt, heads, bname):
    code, tdt = DTYPES[dt]
    nh, d = heads
    H = nh * d
    b = BATCHES[bname]
    T = b.total_tokens
    qkv = _qkv(T, H, 21, dt)
    q = qkv[:, :H].astype(np.float64).reshape(T, nh, d)
    k = qkv[:, H:2 * H].astype(np.float64).reshape(T, nh, d)
    v = qkv[:, 2 * H:].astype(np.float64).reshape(T, nh, d)
    o_ref = oracle.attention_forward(q, k, v, b).reshape(T, H)
    cu = dev_i32(b.cu_seqlens)
    pre = dev_i32(b.prefix_len) if b.mask == "prefix" else None
    t = dev(qkv, dt)
    o = torch.full((T, H), float("nan"), dtype=tdt, device="cuda")
    lse = torch.full((T, nh), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_attention_fwd(code, t, o, lse, cu, pre, T, b.num_seqs, b.max_seqlen, H, nh)
    sync()
    assert rel_l2(host(o), o_ref) < TOL[dt] / 2
    assert rel_l2(host(lse), _lse_ref(q, k, b)) < 1e-5

    # backward, with and without the inverse rotation of dq, dk; bf16 with
    # dq recomputing the softmax gradient and with dq reading it stored
    do = rnd((T, H), 22, dt=dt)
    dq, dk, dv = oracle.attention_backward(q, k, v, do.astype(np.float64).reshape(T, nh, d), b)
    pre_h = b.prefix_len if b.mask == "prefix" else None
    for r, stored in [(0, False), (d // 2, False)] + ([(0, True), (d // 2, True)] if dt == "bf16" else []):
        dqr, dkr = dq, dk
        pos = ct = st = None
        if r:
            p = oracle.positions(b.cu_seqlens)
            cos, sin = oracle.rope_tables(p, r, 10000.0)
            dqr = oracle.rope(dq, cos, sin, r, inverse=True)
            dkr = oracle.rope(dk, cos, sin, r, inverse=True)
            pos = torch.empty(T, dtype=torch.int32, device="cuda")
            ct = torch.empty(b.max_seqlen * r // 2, dtype=torch.float32, device="cuda")
            st = torch.empty_like(ct)
            scratch = torch.zeros((T, 3 * H), dtype=tdt, device="cuda")  # rope on a scratch copy fills the tables
            F.fl_test_rope(code, scratch, cu, b.num_seqs, T, b.max_seqlen, H, nh, r, 10000.0, pos, ct, st)
        dqkv = torch.full((T, 3 * H), float("nan"), dtype=tdt, device="cuda")
        delta = torch.empty((T, nh), dtype=torch.float32, device="cuda")
        ds = _ds_work(b.cu_seqlens, pre_h, nh) if stored else None
        F.fl_test_attention_bwd(code, t, o, lse, dev(do, dt), dqkv, delta, cu, pre, pos, ct, st, r, T, b.num_seqs,
                                b.max_seqlen, H, nh, ds_work=ds)
        sync()
        g = host(dqkv)
        tol = TOL[dt] / 2
        assert rel_l2(g[:, :H], dqr.reshape(T, H)) < tol, (r, stored)
        assert rel_l2(g[:, H:2 * H], dkr.reshape(T, H)) < tol, (r, stored)
        assert rel_l2(g[:, 2 * H:], dv.reshape(T, H)) < tol, (r, stored)


@pytest.mark.parametrize("stored", [False, True])
@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_attention_long_sequence(mask, stored):
    """One 8192-token sequence (bf16, 2 heads of 128; prefix-LM with a
    2048-token context), forward and backward with the inverse rotation; dq
    from the recomputed or the stored softmax gradient."""
    nh, d = 2, 128
    H, T = nh * d, 8192
    b = synth.Batch(np.array([0, T], np.int32), np.array([0, 1], np.int32), mask,
                    np.array([2048], np.int32) if mask == "prefix" else None)
    qkv = _qkv(T, H, 23, "bf16")
    q = qkv[:, :H].astype(np.float64).reshape(T, nh, d)
    k = qkv[:, H:2 * H].astype(np.float64).reshape(T, nh, d)
    v = qkv[:, 2 * H:].astype(np.float64).reshape(T, nh, d)
    cu = dev_i32(b.cu_seqlens)
    pre = dev_i32(b.prefix_len) if mask == "prefix" else None
    t = dev(qkv, "bf16")
    o = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((T, nh), dtype=torch.float32, device="cuda")
    F.fl_test_attention_fwd(F.FL_BF16, t, o, lse, cu, pre, T, 1, T, H, nh)
    r = d // 2
    pos = torch.empty(T, dtype=torch.int32, device="cuda")
    ct = torch.empty(T * r // 2, dtype=torch.float32, device="cuda")
    st = torch.empty_like(ct)
    F.fl_test_rope(F.FL_BF16, torch.zeros((T, 3 * H), dtype=torch.bfloat16, device="cuda"), cu, 1, T, T, H, nh, r,
                   10000.0, pos, ct, st)
    do = rnd((T, H), 24, dt="bf16")
    dqkv = torch.empty((T, 3 * H), dtype=torch.bfloat16, device="cuda")
    delta = torch.empty((T, nh), dtype=torch.float32, device="cuda")
    ds = _ds_work(b.cu_seqlens, b.prefix_len if mask == "prefix" else None, nh) if stored else None
    F.fl_test_attention_bwd(F.FL_BF16, t, o, lse, dev(do, "bf16"), dqkv, delta, cu, pre, pos, ct, st, r, T, 1, T,
                            H, nh, ds_work=ds)
    sync()
    assert rel_l2(host(o), oracle.attention_forward(q, k, v, b).reshape(T, H)) < TOL["bf16"] / 2
    dq, dk, dv = oracle.attention_backward(q, k, v, do.astype(np.float64).reshape(T, nh, d), b)
    cos, sin = oracle.rope_tables(oracle.positions(b.cu_seqlens), r, 10000.0)
    g = host(dqkv)
    assert rel_l2(g[:, :H], oracle.rope(dq, cos, sin, r, inverse=True).reshape(T, H)) < TOL["bf16"] / 2
    assert rel_l2(g[:, H:2 * H], oracle.rope(dk, cos, sin, r, inverse=True).reshape(T, H)) < TOL["bf16"] / 2
    assert rel_l2(g[:, 2 * H:], dv.reshape(T, H)) < TOL["bf16"] / 2


def test_attention_stored_ds_deterministic_and_checked():
    """bf16 backward with the stored softmax gradient: two calls give the same
    bits, the result agrees with the recomputing dq, and a ds_work one tile
    short is refused (FL_ERR_WORKSPACE) before any tile is written."""
    nh, d = 4, 128
    H = nh * d
    b = BATCHES["ragged_prefix"]
    T, S = b.total_tokens, b.num_seqs
    t = dev(_qkv(T, H, 31, "bf16"), "bf16")
    cu, pre = dev_i32(b.cu_seqlens), dev_i32(b.prefix_len)
    o = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((T, nh), dtype=torch.float32, device="cuda")
    F.fl_test_attention_fwd(F.FL_BF16, t, o, lse, cu, pre, T, S, b.max_seqlen, H, nh)
    do = dev(rnd((T, H), 32), "bf16")
    delta = torch.empty((T, nh), dtype=torch.float32, device="cuda")
    outs = []
    for stored in (True, True, False):
        dqkv = torch.full((T, 3 * H), float("nan"), dtype=torch.bfloat16, device="cuda")
        ds = _ds_work(b.cu_seqlens, b.prefix_len, nh) if stored else None
        F.fl_test_attention_bwd(F.FL_BF16, t, o, lse, do, dqkv, delta, cu, pre, None, None, None, 0, T, S,
                                b.max_seqlen, H, nh, ds_work=ds)
        sync()
        outs.append(host(dqkv))
    assert np.array_equal(outs[0], outs[1])
    assert rel_l2(outs[0][:, :H], outs[2][:, :H]) < 1e-2
    assert np.array_equal(outs[0][:, H:], outs[2][:, H:])  # dk, dv: the same kernel either way
    n = F.fl_test_attention_ds_bytes(b.cu_seqlens, b.prefix_len, nh)
    short = torch.empty(n - 64 * 64 * 2, dtype=torch.uint8, device="cuda")
    dqkv = torch.empty((T, 3 * H), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(F.FlglmError) as e:
        F.fl_test_attention_bwd(F.FL_BF16, t, o, lse, do, dqkv, delta, cu, pre, None, None, None, 0, T, S,
                                b.max_seqlen, H, nh, ds_work=short)
    assert e.value.code == F.FL_ERR_WORKSPACE


# ---------------------------------------------------------------------------
# P-tuning v2 prefix keys / values (Appendix A, P-tuning v2 section)
# ---------------------------------------------------------------------------

def _lse_prefix_ref(q, k, pk, b):
    """Natural-log sum-exp of the scaled scores over every key a query sees:
    the whole prefix plus its visible own keys."""
    T, nh, d = q.shape
    out = np.zeros((T, nh))
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        L = r1 - r0
        P = None if b.mask != "prefix" else int(b.prefix_len[s])
        allowed = np.concatenate([np.ones((L, len(pk)), bool), oracle.allowed_mask(L, P)], axis=1)
        for h in range(nh):
            S = (q[r0:r1, h] @ np.concatenate([pk[:, h], k[r0:r1, h]]).T) / math.sqrt(d)
            S = np.where(allowed, S, -np.inf)
            m = S.max(axis=1, keepdims=True)
            out[r0:r1, h] = (m + np.log(np.exp(S - m).sum(1, keepdims=True)))[:, 0]
    return out


@pytest.mark.parametrize("heads", [(2, 128), (4, 64)])
@pytest.mark.parametrize("bname", list(BATCHES))
@pytest.mark.parametrize("num_prefix", [1, 64, 70])
def test_attention_prefix_fwd_bwd(heads, bname, num_prefix):
    """bf16 attention with num_prefix prefix keys / values in front of every
    sequence: o, LSE, dq / dk / dv (with and without the inverse rotation)
    and the prefix gradients summed over the sequences, against the oracle."""
    nh, d = heads
    H = nh * d
    b = BATCHES[bname]
    T, S = b.total_tokens, b.num_seqs
    qkv = _qkv(T, H, 50 + num_prefix, "bf16")
    pk, pv = rnd((num_prefix, H), 51), rnd((num_prefix, H), 52)
    q = qkv[:, :H].astype(np.float64).reshape(T, nh, d)
    k = qkv[:, H:2 * H].astype(np.float64).reshape(T, nh, d)
    v = qkv[:, 2 * H:].astype(np.float64).reshape(T, nh, d)
    pk3, pv3 = pk.astype(np.float64).reshape(-1, nh, d), pv.astype(np.float64).reshape(-1, nh, d)
    o_ref = oracle.attention_forward(q, k, v, b, pk3, pv3).reshape(T, H)
    cu = dev_i32(b.cu_seqlens)
    pre = dev_i32(b.prefix_len) if b.mask == "prefix" else None
    t, tpk, tpv = dev(qkv, "bf16"), dev(pk, "bf16"), dev(pv, "bf16")
    o = torch.full((T, H), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((T, nh), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_attention_fwd(F.FL_BF16, t, o, lse, cu, pre, T, S, b.max_seqlen, H, nh, tpk, tpv, num_prefix)
    sync()
    assert rel_l2(host(o), o_ref) < TOL["bf16"] / 2
    assert rel_l2(host(lse), _lse_prefix_ref(q, k, pk3, b)) < 1e-5

    do = rnd((T, H), 53)
    dq, dk, dv, dpk, dpv = oracle.attention_backward(q, k, v, do.astype(np.float64).reshape(T, nh, d), b, pk3, pv3)
    pre_h = b.prefix_len if b.mask == "prefix" else None
    for r, stored in [(0, False), (d // 2, False), (0, True), (d // 2, True)]:
        dqr, dkr = dq, dk
        pos = ct = st = None
        if r:
            p = oracle.positions(b.cu_seqlens)
            cos, sin = oracle.rope_tables(p, r, 10000.0)
            dqr = oracle.rope(dq, cos, sin, r, inverse=True)
            dkr = oracle.rope(dk, cos, sin, r, inverse=True)
            pos = torch.empty(T, dtype=torch.int32, device="cuda")
            ct = torch.empty(b.max_seqlen * r // 2, dtype=torch.float32, device="cuda")
            st = torch.empty_like(ct)
            scratch = torch.zeros((T, 3 * H), dtype=torch.bfloat16, device="cuda")
            F.fl_test_rope(F.FL_BF16, scratch, cu, S, T, b.max_seqlen, H, nh, r, 10000.0, pos, ct, st)
        dqkv = torch.full((T, 3 * H), float("nan"), dtype=torch.bfloat16, device="cuda")
        delta = torch.empty((T, nh), dtype=torch.float32, device="cuda")
        part = torch.full((2, S, num_prefix, H), float("nan"), dtype=torch.float32, device="cuda")
        ds = _ds_work(b.cu_seqlens, pre_h, nh, num_prefix) if stored else None
        F.fl_test_attention_bwd(F.FL_BF16, t, o, lse, dev(do, "bf16"), dqkv, delta, cu, pre, pos, ct, st, r, T, S,
                                b.max_seqlen, H, nh, tpk, tpv, num_prefix, part, ds_work=ds)
        sync()
        g = host(dqkv)
        tol = TOL["bf16"] / 2
        assert rel_l2(g[:, :H], dqr.reshape(T, H)) < tol, (r, stored)
        assert rel_l2(g[:, H:2 * H], dkr.reshape(T, H)) < tol, (r, stored)
        assert rel_l2(g[:, 2 * H:], dv.reshape(T, H)) < tol, (r, stored)
        pg = host(part).sum(axis=1)  # sequence partials -> the batch's prefix gradients
        assert rel_l2(pg[0], dpk.reshape(-1, H)) < tol, (r, stored)
        assert rel_l2(pg[1], dpv.reshape(-1, H)) < tol, (r, stored)


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_attention_offsets_past_2_31_bytes(mask):
    """One 90037-token sequence at the ChatGLM-6B width (32 heads of 128,
    q|k|v rows of 24 KB, so the sequence spans 2.2 GB and its late tiles sit
    past 2^31 bytes), with a 70-row P-tuning prefix and the inverse rotation.
    The output gradient is zero except on a few rows at the start, middle and
    end, so the oracle's few-rows attention gives the whole dk, dv and prefix
    gradients; o, lse and dq are compared on those rows, and dq of every other
    row must be exactly zero."""
    nh, d, Lp = 32, 128, 70
    H, L = nh * d, 90037
    r = d // 2
    P = L // 4 if mask == "prefix" else None
    gen = torch.Generator(device="cuda").manual_seed(90037)
    t = torch.randn((L, 3 * H), generator=gen, device="cuda").to(torch.bfloat16)
    tpk = torch.randn((Lp, H), generator=gen, device="cuda").to(torch.bfloat16)
    tpv = torch.randn((Lp, H), generator=gen, device="cuda").to(torch.bfloat16)
    rows = np.unique(np.concatenate([[0, 1, 2, 63, 64, L // 2, P or 5], np.arange(L - 64, L)]))
    do_rows = torch.randn((len(rows), H), generator=gen, device="cuda").to(torch.bfloat16)
    tdo = torch.zeros((L, H), dtype=torch.bfloat16, device="cuda")
    tdo[torch.from_numpy(rows).cuda()] = do_rows
    assert L * 3 * H * 2 > (1 << 31)
    cu = dev_i32(np.array([0, L]))
    pre = dev_i32(np.array([P])) if P is not None else None
    o = torch.full((L, H), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((L, nh), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_attention_fwd(F.FL_BF16, t, o, lse, cu, pre, L, 1, L, H, nh, tpk, tpv, Lp)
    pos = torch.empty(L, dtype=torch.int32, device="cuda")
    ct = torch.empty(L * r // 2, dtype=torch.float32, device="cuda")
    st = torch.empty_like(ct)
    F.fl_test_rope(F.FL_BF16, torch.zeros((L, 3 * H), dtype=torch.bfloat16, device="cuda"), cu, 1, L, L, H, nh, r,
                   10000.0, pos, ct, st)
    dqkv = torch.full((L, 3 * H), float("nan"), dtype=torch.bfloat16, device="cuda")
    delta = torch.empty((L, nh), dtype=torch.float32, device="cuda")
    part = torch.full((2, 1, Lp, H), float("nan"), dtype=torch.float32, device="cuda")
    F.fl_test_attention_bwd(F.FL_BF16, t, o, lse, tdo, dqkv, delta, cu, pre, pos, ct, st, r, L, 1, L, H, nh,
                            tpk, tpv, Lp, part)
    sync()
    qkv = host(t)
    q, k, v = (qkv[:, i * H:(i + 1) * H].reshape(L, nh, d) for i in range(3))
    pk, pv = host(tpk).reshape(Lp, nh, d), host(tpv).reshape(Lp, nh, d)
    o_r, lse_r, dq_r, dk_r, dv_r, dpk, dpv = oracle.attention_query_rows(
        q, k, v, rows, P, pk, pv, host(do_rows).reshape(-1, nh, d))
    cos, sin = oracle.rope_tables(np.arange(L), r, 10000.0)
    tol = TOL["bf16"] / 2
    errs = {"o": rel_l2(host(o[torch.from_numpy(rows).cuda()]), o_r.reshape(-1, H)),
            "lse": rel_l2(host(lse[torch.from_numpy(rows).cuda()]), lse_r)}
    g = host(dqkv)
    errs["dq"] = rel_l2(g[rows, :H], oracle.rope(dq_r, cos[rows], sin[rows], r, inverse=True).reshape(-1, H))
    errs["dk"] = rel_l2(g[:, H:2 * H], oracle.rope(dk_r, cos, sin, r, inverse=True).reshape(L, H))
    errs["dv"] = rel_l2(g[:, 2 * H:], dv_r.reshape(L, H))
    pg = host(part)
    errs["dprefix_k"] = rel_l2(pg[0, 0], dpk.reshape(Lp, H))
    errs["dprefix_v"] = rel_l2(pg[1, 0], dpv.reshape(Lp, H))
    print(f"[attention L={L} {mask}] {errs}", flush=True)
    assert errs["lse"] < 1e-5
    assert all(e < tol for e in errs.values()), errs
    quiet = np.ones(L, bool)
    quiet[rows] = False
    assert (g[quiet, :H] == 0).all()
