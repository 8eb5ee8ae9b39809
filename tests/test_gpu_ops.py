"""Kernel-level parity: each HIP kernel (through sgd_ops.h) against the oracle's definition of
the same operation, on seeded inputs spanning several tiles and ragged tails."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle.numerics import decode, round_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_29505_amd as P
    P.lib()
    return P


def dev(arr):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).cuda()


def host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return decode(t.view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    return t.cpu().numpy().astype(np.float64)


def empty(shape, dtype):
    import torch
    return torch.full(shape, float("nan"), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")


def relmax(x, ref):
    return float(np.max(np.abs(x - ref)) / np.max(np.abs(ref)))


TILES = [0, 1, 2, 3, 4, 5]
TILE_WIDTH = {1: 256, 2: 128, 3: 256, 4: 128, 5: 192}


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("M,N,K", [(200, 256, 128), (300, 768, 192), (64, 1024, 64), (1000, 512, 320), (513, 1024, 448),
                                   (130, 200, 64), (257, 580, 128)])
def test_linear_bf16(P, M, N, K, tile):
    rng = np.random.default_rng(M + N + K)
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), "bf16")
    b = synth.representable(0.1 * rng.standard_normal(N), "bf16")
    out = empty((M, N), "bf16")
    P.op_linear(dev(A), dev(W), out, bias=dev(b), tile=tile)
    ref = decode(A, "bf16") @ decode(W, "bf16").T + b
    got = host(out)
    assert np.isfinite(got).all()
    assert np.max(np.abs(got - round_bf16(ref))) <= 2 ** -7 * np.max(np.abs(ref))


@pytest.mark.parametrize("act", [1, 2, 3])
def test_linear_act_bf16(P, act):
    rng = np.random.default_rng(act)
    M, N, K = 130, 256, 192
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), "bf16")
    out = empty((M, N), "bf16")
    P.op_linear(dev(A), dev(W), out, act=act)
    z = decode(A, "bf16") @ decode(W, "bf16").T
    f = {1: om.gelu_erf, 2: om.gelu_tanh, 3: om.silu}[act]
    ref = f(z)
    assert relmax(host(out), ref) <= 1e-2


@pytest.mark.parametrize("tile", TILES)
def test_linear_gated_bf16(P, tile):
    rng = np.random.default_rng(11 + tile)
    # gate and up halves split evenly over the tiles: 2F a multiple of the tile width
    M, F, K = 260, (288 if tile == 5 else 256), 128
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((2 * F, K)) / np.sqrt(K), "bf16")
    b = synth.representable(0.1 * rng.standard_normal(2 * F), "bf16")
    out = empty((M, F), "bf16")
    P.op_linear(dev(A), dev(W), out, bias=dev(b), act=3, gated=True, tile=tile)
    z = decode(A, "bf16") @ decode(W, "bf16").T + b
    ref = om.silu(z[:, :F]) * z[:, F:]
    assert relmax(host(out), ref) <= 1e-2


def test_linear_row_tail_split_bf16(P):
    """8256 = 32 x 258 rows (U-ViT batch): the automatic tiling runs rows [0, 8192) and the
    64-row tail as two launches; both must index rows globally."""
    rng = np.random.default_rng(8256)
    M, N, K = 8256, 4096, 128
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), "bf16")
    b = synth.representable(0.1 * rng.standard_normal(N), "bf16")
    out = empty((M, N), "bf16")
    P.op_linear(dev(A), dev(W), out, bias=dev(b), act=1)
    ref = om.gelu_erf(decode(A, "bf16") @ decode(W, "bf16").T + b)
    got = host(out)
    assert np.isfinite(got).all()
    assert relmax(got, ref) <= 1e-2
    assert relmax(got[8192:], ref[8192:]) <= 1e-2


def test_residual_row_tail_split_bf16(P):
    """Residual epilogue with per-sample gates (258 rows per sample) across the row-tail split."""
    rng = np.random.default_rng(258)
    B, ntok, N, K = 32, 258, 4096, 128
    M = B * ntok
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), "bf16")
    b = synth.representable(0.1 * rng.standard_normal(N), "bf16")
    h0 = rng.standard_normal((M, N)).astype(np.float32)
    d0 = rng.standard_normal((M, N)).astype(np.float32)
    gate = rng.standard_normal((B, N)).astype(np.float32)
    th, td = dev(h0), dev(d0)
    P.op_residual(dev(A), dev(W), th, bias=dev(b), delta=td, delta_mode=2, gate=dev(gate), ntok=ntok)
    v = (decode(A, "bf16") @ decode(W, "bf16").T + b) * np.repeat(gate, ntok, axis=0)
    assert relmax(host(th), h0 + v) <= 1e-3
    assert relmax(host(td), d0 + v) <= 1e-3


@pytest.mark.parametrize("M,N,K", [(72, 128, 64), (256, 768, 256), (144, 1024, 256)])
def test_linear_f32(P, M, N, K):
    rng = np.random.default_rng(M * N)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32)
    out = empty((M, N), "f32")
    P.op_linear(dev(A), dev(W), out)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    assert relmax(host(out), ref) <= 1e-5


def _heads_inputs(rng, B, H, nq, nk, dh, dtype, npq, npk):
    q = rng.standard_normal((B * H, npq, dh)) * 1.5
    k = rng.standard_normal((B * H, npk, dh)) * 1.5
    v = rng.standard_normal((B * H, npk, dh))
    qs, ks, vs = synth.store(q, dtype), synth.store(k, dtype), synth.store(v, dtype)
    vts = np.ascontiguousarray(vs.transpose(0, 2, 1))
    return qs, ks, vs, vts


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,H,nq,nk,dh", [(1, 2, 200, 200, 128), (2, 3, 80, 80, 72), (2, 2, 66, 66, 64),
                                          (2, 2, 96, 77, 64), (1, 1, 256, 256, 64), (1, 2, 130, 1, 64),
                                          # >= 8 key blocks: keys split between two wave halves
                                          # (odd block count, ragged tail, padded head dim)
                                          (1, 2, 300, 600, 128), (1, 3, 150, 1000, 64), (2, 2, 130, 700, 72),
                                          (1, 2, 64, 513, 128),
                                          # many heads: 256-query workgroups (DiT, one per head; a
                                          # ragged case; the SDXL cross-attention shape, 77 keys),
                                          # U-ViT's 258 queries in one workgroup, and 128-query
                                          # workgroups where 256 would add padded queries
                                          (32, 16, 256, 256, 72), (16, 64, 250, 240, 64), (8, 20, 1024, 77, 64),
                                          (32, 16, 258, 258, 64), (16, 64, 300, 300, 64), (16, 32, 260, 200, 128)])
def test_attention(P, dtype, B, H, nq, nk, dh):
    rng = np.random.default_rng(nq * 7 + nk + dh)
    npq, npk = -(-nq // 64) * 64, -(-nk // 64) * 64
    qs, ks, vs, vts = _heads_inputs(rng, B, H, nq, nk, dh, dtype, npq, npk)
    o = empty((B, nq, H * dh), dtype)
    P.op_attention(dev(qs), dev(ks), dev(vts), o, B, H, dh, nq, nk)
    q = decode(qs, dtype)[:, :nq].reshape(B, H, nq, dh)
    k = decode(ks, dtype)[:, :nk].reshape(B, H, nk, dh)
    v = decode(vs, dtype)[:, :nk].reshape(B, H, nk, dh)
    ref = om.merge_heads(om.attention(q, k, v))
    got = host(o)
    assert np.isfinite(got).all()
    tol = 1.5e-2 if dtype == "bf16" else 1e-5
    assert relmax(got, ref) <= tol


@pytest.mark.parametrize("B,H,nq,nk,dh", [(1, 2, 300, 1000, 128), (2, 2, 130, 700, 72), (32, 16, 256, 256, 72),
                                          (2, 2, 96, 77, 64), (16, 64, 300, 300, 64)])
def test_attention_rising_scores(P, B, H, nq, nk, dh):
    """Key norms growing along the sequence: later key blocks keep exceeding the running maximum
    by many binades, so the online softmax raises its reference block after block instead of
    keeping it."""
    rng = np.random.default_rng(nq + 3 * nk + dh)
    npq, npk = -(-nq // 64) * 64, -(-nk // 64) * 64
    q = rng.standard_normal((B * H, npq, dh)) * 1.5
    k = rng.standard_normal((B * H, npk, dh)) * np.linspace(0.1, 8.0, npk)[None, :, None]
    v = rng.standard_normal((B * H, npk, dh))
    qs, ks, vs = synth.store(q, "bf16"), synth.store(k, "bf16"), synth.store(v, "bf16")
    vts = np.ascontiguousarray(vs.transpose(0, 2, 1))
    o = empty((B, nq, H * dh), "bf16")
    P.op_attention(dev(qs), dev(ks), dev(vts), o, B, H, dh, nq, nk)
    qd = decode(qs, "bf16")[:, :nq].reshape(B, H, nq, dh)
    kd = decode(ks, "bf16")[:, :nk].reshape(B, H, nk, dh)
    vd = decode(vs, "bf16")[:, :nk].reshape(B, H, nk, dh)
    ref = om.merge_heads(om.attention(qd, kd, vd))
    got = host(o)
    assert np.isfinite(got).all()
    assert relmax(got, ref) <= 1.5e-2


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind,d,M", [(0, 256, 70), (0, 4096, 70), (1, 1024, 70), (1, 1280, 70), (2, 1152, 70),
                                      # many rows: one wave per row, ragged last workgroup
                                      (0, 256, 4099), (1, 1280, 4099), (2, 1152, 4099),
                                      # many rows of 128-lane multiples: two waves per row
                                      (1, 1024, 4099), (0, 512, 4097), (2, 2048, 4099),
                                      # many rows too wide for two rows per thread group
                                      (0, 8192, 4100)])
def test_norm(P, dtype, kind, d, M):
    rng = np.random.default_rng(kind * 100 + d + M)
    ntok = 35 if M == 70 else 4099
    x = (rng.standard_normal((M, d)) * 3 + 0.5).astype(np.float32)
    w = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    b = (0.1 * rng.standard_normal(d)).astype(np.float32)
    mod = rng.standard_normal((-(-M // ntok), 6 * d)).astype(np.float32)
    y = empty((M, d), dtype)
    x64 = x.astype(np.float64)
    if kind == 0:
        P.op_norm(0, dev(x), y, 1e-5, w=dev(w))
        ref = om.rmsnorm(x64, w)
    elif kind == 1:
        P.op_norm(1, dev(x), y, 1e-5, w=dev(w), b=dev(b))
        ref = om.layernorm(x64, w, b, eps=1e-5)
    else:
        md = dev(mod)
        P.op_norm(2, dev(x), y, 1e-6, shift=md[:, :d], scale=md[:, d:2 * d], ntok=ntok)
        shift = np.repeat(mod[:, :d], ntok, axis=0)[:M]
        scale = np.repeat(mod[:, d:2 * d], ntok, axis=0)[:M]
        ref = om.layernorm(x64, eps=1e-6) * (1 + scale) + shift
    got = host(y)
    if dtype == "bf16":
        assert np.max(np.abs(got - round_bf16(ref))) <= 2 ** -7 * np.max(np.abs(ref))
    else:
        assert relmax(got, ref) <= 1e-5


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind,d,M,r", [(0, 4096, 1024, 1), (0, 4096, 1024, 3), (0, 4096, 1024, 9), (1, 1280, 4099, 2),
                                        (1, 1024, 4099, 5), (2, 1152, 4099, 4), (0, 256, 70, 32), (2, 1152, 70, 7)])
def test_norm_fold_bitwise(P, dtype, kind, d, M, r):
    """The pre-norm that absorbs a frozen run: the stream and the normalised rows bit for bit
    those of the frozen-run pass followed by the plain pre-norm, for runs of 1 to 32 updates
    (loaded in groups, added one at a time in stack order) and every norm kind and row split."""
    import torch
    rng = np.random.default_rng(kind * 1000 + d + M + r)
    ntok = 35 if M == 70 else 4099
    x = (rng.standard_normal((M, d)) * 3 + 0.5).astype(np.float32)
    deltas = [dev((rng.standard_normal((M, d)) * 0.7).astype(np.float32)) for _ in range(r)]
    w = dev((1 + 0.1 * rng.standard_normal(d)).astype(np.float32))
    b = dev((0.1 * rng.standard_normal(d)).astype(np.float32))
    md = dev(rng.standard_normal((-(-M // ntok), 6 * d)).astype(np.float32))
    kw = {"w": w} if kind == 0 else {"w": w, "b": b} if kind == 1 else {"shift": md[:, :d], "scale": md[:, d:2 * d],
                                                                         "ntok": ntok}
    eps = 1e-6 if kind == 2 else 1e-5
    x1, x2 = dev(x), dev(x)
    y1, y2 = empty((M, d), dtype), empty((M, d), dtype)
    P.op_frozen_run(x1.view(-1), [t.view(-1) for t in deltas])
    P.op_norm(kind, x1, y1, eps, **kw)
    P.op_norm_fold(kind, x2, y2, eps, deltas, **kw)
    torch.cuda.synchronize()
    bits = (lambda t: t.view(torch.int16)) if dtype == "bf16" else (lambda t: t.view(torch.int32))
    assert torch.equal(x1.view(torch.int32), x2.view(torch.int32))
    assert torch.equal(bits(y1), bits(y2))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,d,n_out", [(32, 1152, 6912), (2, 1152, 6912), (5, 256, 200), (40, 128, 96), (3, 64, 32),
                                         (8, 1280, 1280), (33, 2048, 100), (4, 1600, 70), (40, 320, 2100),
                                         (3, 64, 2048)])
def test_adaln_mod(P, dtype, B, d, n_out):
    """DiT modulation vectors SiLU(c) W_ada^T + b: fp32 accumulation of the exact products
    (bf16 weights run on the matrix cores with x split into three bf16 parts).  Shapes: DiT,
    the UNet time projection, ragged features and samples, k ranges of several load groups with
    a partial last chunk, and the wide variant (2048 outputs or more) with ragged features,
    more than 32 samples and one or several load groups."""
    rng = np.random.default_rng(B * 7 + d + n_out)
    x = om.silu(rng.standard_normal((B, d))).astype(np.float32)
    W = synth.store(rng.standard_normal((n_out, d)) / np.sqrt(d), dtype)
    b = synth.representable(0.02 * rng.standard_normal(n_out), "f32")
    mod = empty((B, n_out), "f32")
    P.op_adaln_mod(dev(x), dev(W), mod, bias=dev(b))
    ref = x.astype(np.float64) @ decode(W, dtype).T + b
    assert relmax(host(mod), ref) < 2e-6


def test_adaln_mod_wide_widths_bitwise(P):
    """The wide modulation kernel (2048 outputs or more) takes workgroups of eight, four or two
    waves as the grid size allows, and computes every output in the same order whatever the
    width: the rows of a 512-sample problem (eight-wave workgroups) equal those of its 256- and
    32-sample slices (four- and two-wave workgroups) bit for bit."""
    rng = np.random.default_rng(5)
    B, d, n_out = 512, 256, 8192
    x = om.silu(rng.standard_normal((B, d))).astype(np.float32)
    W = synth.store(rng.standard_normal((n_out, d)) / np.sqrt(d), "bf16")
    b = synth.representable(0.02 * rng.standard_normal(n_out), "f32")
    outs = []
    for nb in (512, 256, 32):
        mod = empty((nb, n_out), "f32")
        P.op_adaln_mod(dev(np.ascontiguousarray(x[:nb])), dev(W), mod, bias=dev(b))
        outs.append(host(mod))
    ref = x[:32].astype(np.float64) @ decode(W, "bf16").T + b
    assert relmax(outs[2], ref) < 2e-6
    assert np.array_equal(outs[0][:256], outs[1])
    assert np.array_equal(outs[0][:32], outs[2])


def test_frozen_run_bitwise(P):
    rng = np.random.default_rng(0)
    n = 4096 * 33
    h = rng.standard_normal(n).astype(np.float32)
    ds = [rng.standard_normal(n).astype(np.float32) for _ in range(5)]
    th = dev(h)
    P.op_frozen_run(th, [dev(d) for d in ds])
    ref = h.copy()
    for d in ds:
        ref = (ref + d).astype(np.float32)
    assert np.array_equal(th.cpu().numpy(), ref)


def _tile_cases():
    out = []
    for dtype in ("bf16", "f32"):
        for tile in (TILES if dtype == "bf16" else [0]):
            out.append((dtype, tile))
    return out


@pytest.mark.parametrize("dtype,tile", _tile_cases())
@pytest.mark.parametrize("B,N,H,dh,rope,bias", [(1, 200, 2, 128, True, False), (2, 80, 16, 72, False, True),
                                                (2, 66, 4, 64, False, False), (1, 130, 2, 128, False, True),
                                                (3, 77, 4, 128, True, True),
                                                (2, 90, 6, 64, True, True), (1, 150, 4, 96, True, False),
                                                # rotary tiles that straddle the q/k and k/v boundaries
                                                # and hold part of a head (d = 640, 192 on 256-wide tiles)
                                                (1, 100, 5, 128, True, True), (2, 70, 3, 64, True, False)])
def test_heads(P, dtype, tile, B, N, H, dh, rope, bias):
    if dtype == "f32" and rope:
        pytest.skip("rotary epilogue is bf16 only")
    rng = np.random.default_rng(N + dh)
    d = H * dh
    M = B * N
    np_ = -(-N // 64) * 64
    A = synth.store(rng.standard_normal((M, d)), dtype)
    W = synth.store(rng.standard_normal((3 * d, d)) / np.sqrt(d), dtype)
    b = synth.representable(0.1 * rng.standard_normal(3 * d), dtype) if bias else None
    q, k = empty((B * H, np_, dh), dtype), empty((B * H, np_, dh), dtype)
    vt = empty((B * H, dh, np_), dtype)
    P.op_heads(dev(A), dev(W), q, k, vt, 3, 0, N, H, dh, bias=dev(b) if bias else None, rope=rope, tile=tile)
    z = decode(A, dtype) @ decode(W, dtype).T + (b if bias else 0)
    Q, K, V = (om.heads(z[:, i * d:(i + 1) * d].reshape(B, N, d), H) for i in range(3))
    if rope:
        Q, K = om.rope(Q), om.rope(K)
    got_q = host(q).reshape(B, H, np_, dh)[:, :, :N]
    got_k = host(k).reshape(B, H, np_, dh)[:, :, :N]
    got_v = host(vt).reshape(B, H, dh, np_)[:, :, :, :N].transpose(0, 1, 3, 2)
    tol = 2 ** -7 if dtype == "bf16" else 1e-5
    for g, r in ((got_q, Q), (got_k, K), (got_v, V)):
        assert np.isfinite(g).all()
        assert np.max(np.abs(g - r)) <= tol * np.max(np.abs(r))


@pytest.mark.parametrize("dtype,tile", _tile_cases())
@pytest.mark.parametrize("M,N,K,gated_rows,mode", [(200, 256, 256, 0, 1), (160, 1152, 1152, 80, 2), (130, 512, 1024, 0, 0)])
def test_residual(P, dtype, tile, M, N, K, gated_rows, mode):
    rng = np.random.default_rng(M + K + mode)
    A = synth.store(rng.standard_normal((M, K)), dtype)
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), dtype)
    b = synth.representable(0.1 * rng.standard_normal(N), dtype)
    h0 = rng.standard_normal((M, N)).astype(np.float32)
    d0 = rng.standard_normal((M, N)).astype(np.float32)
    gate = rng.standard_normal((2, 6 * N)).astype(np.float32) if gated_rows else None
    th, td = dev(h0), dev(d0)
    g_dev = dev(gate)[:, 2 * N:3 * N] if gated_rows else None
    P.op_residual(dev(A), dev(W), th, bias=dev(b), delta=td if mode else None, delta_mode=mode, gate=g_dev,
                  ntok=gated_rows or 1, tile=tile)
    v = decode(A, dtype) @ decode(W, dtype).T + b
    if gated_rows:
        v = v * np.repeat(gate[:, 2 * N:3 * N], gated_rows, axis=0)
    tol = 1e-2 if dtype == "bf16" else 1e-5
    assert relmax(host(th), h0 + v) <= tol * 0.1
    if mode == 1:
        assert relmax(host(td), v) <= 1e-5
    elif mode == 2:
        assert relmax(host(td), d0 + v) <= 1e-5
    else:
        assert np.array_equal(host(td), d0.astype(np.float64))


@pytest.mark.parametrize("M,N,K,ks", [(1024, 4096, 12288, 2), (200, 256, 8192, 2), (300, 520, 1024, 4),
                                      (64, 128, 512, 8)])
def test_linear_split(P, M, N, K, ks):
    """K ranges of a residual projection (the split MLP output GEMM): part s is the exact-product
    fp32 sum over columns [s K / ks, (s + 1) K / ks), the bias in part 0 only; the LLaDA-8B
    shape, ragged rows and columns, four and eight ranges."""
    rng = np.random.default_rng(M + N + K + ks)
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((N, K)) / np.sqrt(K), "bf16")
    b = synth.representable(0.1 * rng.standard_normal(N), "f32")
    parts = empty((ks, M, N), "f32")
    P.op_linear_split(dev(A), dev(W), parts, bias=dev(b))
    got = host(parts)
    a64, w64 = decode(A, "bf16"), decode(W, "bf16")
    kr = K // ks
    for s in range(ks):
        ref = a64[:, s * kr:(s + 1) * kr] @ w64[:, s * kr:(s + 1) * kr].T + (b if s == 0 else 0.0)
        assert relmax(got[s], ref) < 1e-5, s


def test_linear_split_refuses_bad_ranges(P):
    import torch
    A = torch.zeros((64, 640), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((128, 640), dtype=torch.bfloat16, device="cuda")
    for ks in (1, 3, 9):  # one range, K not a multiple of 64 ks, too many ranges
        parts = torch.zeros((ks, 64, 128), dtype=torch.float32, device="cuda")
        with pytest.raises(P.SgdError):
            P.op_linear_split(A, W, parts)


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("tile", TILES)
def test_heads_kv_only(P, tile, rope):
    """Key/value projection of a context (which0 = 1): columns [0, d) are k, [d, 2d) are v^T;
    with rope, the k columns are read in rotary-pair order."""
    rng = np.random.default_rng(77 + tile)
    B, N, H, dh, K = 3, 77, 5, 64, 192
    d = H * dh
    M = B * N
    np_ = -(-N // 64) * 64
    A = synth.store(rng.standard_normal((M, K)), "bf16")
    W = synth.store(rng.standard_normal((2 * d, K)) / np.sqrt(K), "bf16")
    k, vt = empty((B * H, np_, dh), "bf16"), empty((B * H, dh, np_), "bf16")
    P.op_heads(dev(A), dev(W), None, k, vt, 2, 1, N, H, dh, rope=rope, tile=tile)
    z = decode(A, "bf16") @ decode(W, "bf16").T
    Kr, Vr = (om.heads(z[:, i * d:(i + 1) * d].reshape(B, N, d), H) for i in range(2))
    if rope:
        Kr = om.rope(Kr)
    got_k = host(k).reshape(B, H, np_, dh)[:, :, :N]
    got_v = host(vt).reshape(B, H, dh, np_)[:, :, :, :N].transpose(0, 1, 3, 2)
    for g, r in ((got_k, Kr), (got_v, Vr)):
        assert np.isfinite(g).all()
        assert np.max(np.abs(g - r)) <= 2 ** -7 * np.max(np.abs(r))
