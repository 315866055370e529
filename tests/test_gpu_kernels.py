"""Single-kernel parity on the GPU: GEMM epilogues, prefill attention and
RMSNorm against float64 references of the same operation (the oracle's
functions where it has them)."""
import numpy as np
import pytest

from oracle.llama import apply_rope, attention, rms_norm, rope_angles, silu
from workloads import gen
from tests import gpu_util as G

pytestmark = pytest.mark.gpu


def _hs():
    from paper_2502_15524_amd import hs
    return hs


GEMM_SHAPES = [(1, 256, 256), (7, 768, 256), (16, 1376, 256), (33, 512, 688),
               (64, 4096, 4096), (65, 1024, 1024), (200, 768, 256), (512, 1024, 512),
               (777, 1376, 688), (1024, 4096, 4096),
               (12, 16384, 256), (16, 6144, 512),   # wide 9-16-token decode variants
               (3, 2048, 11008), (14, 1024, 5120),  # eight-wave splits of a long k
               (512, 22016, 256), (512, 12288, 256),  # one round of 192 x 256, 192 x 128 tiles
               (4, 73728, 256), (3, 36864, 320),    # LM-head-wide: 8 and 4 row tiles, 2 waves
               (9, 5120, 256), (5, 24576, 192),     # o/down wider than the CUs; 4-tile gate/up
               (8, 4096, 1024),                     # sixteen waves (o projection rule)
               (3, 12288, 512)]                     # three row tiles, one workgroup per CU


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("epi", ["store", "resid", "swiglu", "f32"])
def test_gemm(M, N, K, epi):
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(M * 7 + N + K)
    X = gen.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    Wt = gen.round_to_bf16((rng.standard_normal((N, K)) * 0.05).astype(np.float32))
    acc = X.astype(np.float64) @ Wt.astype(np.float64).T
    kp = -(-K // 64) * 64
    Xp = np.zeros((M, kp), np.float32)     # columns past K are zero
    Xp[:, :K] = X
    dX = G.to_dev_bf16(Xp)
    wt = G.tile_bits(gen.to_bf16_bits(Wt))
    dW = torch.from_numpy(wt.view(np.int16)).cuda()
    if epi == "f32":
        Y = torch.zeros((M, N), dtype=torch.float32, device="cuda")
        ref = acc
    elif epi == "swiglu":
        Y = torch.zeros((M, N // 2), dtype=torch.bfloat16, device="cuda")
        idx = np.arange(N // 2)
        gate = acc[:, (idx // 16) * 32 + idx % 16]
        up = acc[:, (idx // 16) * 32 + 16 + idx % 16]
        ref = silu(gate) * up
    elif epi == "resid":
        R = gen.round_to_bf16(rng.standard_normal((M, N)).astype(np.float32))
        Y = G.to_dev_bf16(R)           # in place: Y = R + X W^T
        ref = R + acc
    else:
        Y = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
        ref = acc
    ldy = Y.shape[1]
    hs.hs_k_gemm(dX.data_ptr(), kp, dW.data_ptr(), Y.data_ptr(), ldy,
                 Y.data_ptr() if epi == "resid" else 0, ldy, M, N, K, epi, G.stream_ptr())
    torch.cuda.synchronize()
    out = Y.cpu().numpy() if epi == "f32" else G.from_dev_bf16(Y)
    scale = np.abs(ref).max()
    err = np.abs(out - ref).max()
    tol = (1e-5 if epi == "f32" else 8e-3) * scale
    assert err <= tol, (err, scale)


@pytest.mark.parametrize("M,N,K", [(16, 4096, 4096), (8, 4096, 11008), (13, 2048, 1024)])
def test_gemm_staged_activations_bitwise(M, N, K):
    """The decode GEMM with its activations staged through LDS as whole rows
    (XS) feeds the MFMAs the same operands as the direct fragment loads: the
    results are bitwise equal (forced through the tuning knob)."""
    import os
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(M + N + K)
    X = gen.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    Wt = gen.round_to_bf16((rng.standard_normal((N, K)) * 0.05).astype(np.float32))
    R = gen.round_to_bf16(rng.standard_normal((M, N)).astype(np.float32))
    dX = G.to_dev_bf16(X)
    dW = torch.from_numpy(G.tile_bits(gen.to_bf16_bits(Wt)).view(np.int16)).cuda()
    outs = []
    old = os.environ.get("HS_SKINNY_CFG")
    try:
        for xs in (0, 1):
            os.environ["HS_SKINNY_CFG"] = f"1,1,16,{xs}"
            Y = G.to_dev_bf16(R)
            hs.hs_k_gemm(dX.data_ptr(), K, dW.data_ptr(), Y.data_ptr(), N, Y.data_ptr(), N,
                         M, N, K, "resid", G.stream_ptr())
            torch.cuda.synchronize()
            outs.append(G.from_dev_bf16(Y))
    finally:
        if old is None:
            os.environ.pop("HS_SKINNY_CFG", None)
        else:
            os.environ["HS_SKINNY_CFG"] = old
    assert np.array_equal(outs[0], outs[1])
    ref = R + X.astype(np.float64) @ Wt.astype(np.float64).T
    assert np.abs(outs[1] - ref).max() <= 8e-3 * np.abs(ref).max()


# 7B-shape projections at a 512-token prompt: few output tiles, so their k
# ranges are split across workgroups (stream-K). Rows are sampled for the
# float64 reference; two calls must agree bitwise.
@pytest.mark.parametrize("N,K,epi", [(12288, 4096, "store"), (4096, 4096, "resid"),
                                     (22016, 4096, "swiglu"), (4096, 11008, "resid")])
def test_gemm_split_k_shapes(N, K, epi):
    torch = G.torch()
    hs = _hs()
    M = 512
    rng = np.random.default_rng(N + K)
    X = gen.round_to_bf16(rng.standard_normal((M, K)).astype(np.float32))
    Wt = gen.round_to_bf16((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
    dX = G.to_dev_bf16(X)
    dW = torch.from_numpy(G.tile_bits(gen.to_bf16_bits(Wt)).view(np.int16)).cuda()
    ncol = N // 2 if epi == "swiglu" else N
    R = gen.round_to_bf16(rng.standard_normal((M, ncol)).astype(np.float32))
    outs = []
    for _ in range(2):
        Y = G.to_dev_bf16(R) if epi == "resid" else torch.zeros((M, ncol), dtype=torch.bfloat16, device="cuda")
        hs.hs_k_gemm(dX.data_ptr(), K, dW.data_ptr(), Y.data_ptr(), ncol,
                     Y.data_ptr() if epi == "resid" else 0, ncol, M, N, K, epi, G.stream_ptr())
        torch.cuda.synchronize()
        outs.append(G.from_dev_bf16(Y))
    assert np.array_equal(outs[0], outs[1])
    rows = np.sort(rng.choice(M, 24, replace=False))
    acc = X[rows].astype(np.float64) @ Wt.astype(np.float64).T
    if epi == "swiglu":
        idx = np.arange(ncol)
        ref = silu(acc[:, (idx // 16) * 32 + idx % 16]) * acc[:, (idx // 16) * 32 + 16 + idx % 16]
    elif epi == "resid":
        ref = R[rows] + acc
    else:
        ref = acc
    err = np.abs(outs[0][rows] - ref).max()
    assert err <= 8e-3 * np.abs(ref).max(), err


@pytest.mark.parametrize("lens,nh,nkv,d", [
    ([1], 4, 4, 64), ([5, 64, 65], 4, 2, 64), ([130, 7, 300], 4, 4, 128),
    ([257], 8, 2, 128), ([64, 128, 1, 33], 2, 1, 128),
    ([1024, 1024], 32, 8, 128),      # enough 128-query tiles for the 8-wave variant
    # 4-wave tiles that do not fit one workgroup per CU (no key split):
    # workgroup counts 512 and 380 (D = 128), 320 and 276 (D = 64), so both
    # multiples of 8 and others
    ([1024], 32, 8, 128), ([1000, 150], 20, 5, 128), ([900, 300], 16, 4, 64),
    ([1000, 400], 12, 6, 64)])
def test_attn_prefill(lens, nh, nkv, d):
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(sum(lens) + nh + d)
    T = sum(lens)
    qkv = gen.round_to_bf16((rng.standard_normal((T, (nh + 2 * nkv) * d)) * 1.5).astype(np.float32))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    dq = G.to_dev_bf16(qkv)
    out = torch.zeros((T, nh * d), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_attn_prefill(dq.data_ptr(), out.data_ptr(), list(cu), nh, nkv, d, G.stream_ptr())
    torch.cuda.synchronize()
    got = G.from_dev_bf16(out)
    q = qkv[:, :nh * d].reshape(T, nh, d).astype(np.float64)
    k = qkv[:, nh * d:(nh + nkv) * d].reshape(T, nkv, d).astype(np.float64)
    v = qkv[:, (nh + nkv) * d:].reshape(T, nkv, d).astype(np.float64)
    for i, n in enumerate(lens):
        s = slice(cu[i], cu[i + 1])
        ref = attention(q[s], k[s], v[s], np.arange(n), np.arange(n))
        err = np.abs(got[s] - ref).max()
        assert err <= 2e-2 * np.abs(ref).max() + 1e-3, (i, err)


def test_attn_prefill_value_ones_gives_ones():
    """V = 1 everywhere: every output is exactly a softmax row sum."""
    torch = G.torch()
    hs = _hs()
    nh, nkv, d, lens = 4, 4, 128, [3, 100, 64]
    T = sum(lens)
    rng = np.random.default_rng(1)
    qkv = np.ones((T, (nh + 2 * nkv) * d), np.float32)
    qkv[:, :2 * nh * d] = rng.standard_normal((T, 2 * nh * d)) * 3
    dq = G.to_dev_bf16(qkv)
    out = torch.zeros((T, nh * d), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_attn_prefill(dq.data_ptr(), out.data_ptr(), [0, 3, 103, 167], nh, nkv, d,
                         G.stream_ptr())
    torch.cuda.synchronize()
    got = G.from_dev_bf16(out)
    assert np.max(np.abs(got - 1.0)) <= 2 ** -7


def _paged_case(lens, nh, nkv, d, seed):
    """Random post-RoPE keys/values of ragged sequences scattered over a KV
    pool [blocks][K|V][nkv][16][d] in a shuffled block order."""
    rng = np.random.default_rng(seed)
    nblk = [-(-n // 16) for n in lens]
    total = sum(nblk) + 3
    perm = rng.permutation(total)
    pool = np.zeros((total, 2, nkv, 16, d), np.float32)
    mb = max(nblk)
    table = np.zeros((len(lens), mb), np.int32)
    ks, vs = [], []
    nxt = 0
    for i, n in enumerate(lens):
        k = gen.round_to_bf16((rng.standard_normal((n, nkv, d)) * 1.5).astype(np.float32))
        v = gen.round_to_bf16(rng.standard_normal((n, nkv, d)).astype(np.float32))
        ks.append(k)
        vs.append(v)
        for bi in range(nblk[i]):
            phys = perm[nxt]
            nxt += 1
            table[i, bi] = phys
            seg = slice(bi * 16, min(n, bi * 16 + 16))
            cnt = seg.stop - seg.start
            pool[phys, 0, :, :cnt] = k[seg].transpose(1, 0, 2)
            pool[phys, 1, :, :cnt] = v[seg].transpose(1, 0, 2)
    q = gen.round_to_bf16((rng.standard_normal((len(lens), nh * d)) * 1.5).astype(np.float32))
    return q, pool, table, ks, vs


@pytest.mark.parametrize("lens,nh,nkv,d", [
    ([2100] + [int(x) for x in np.random.default_rng(3).integers(900, 2000, 15)], 32, 8, 128),
    ([600, 2000, 17, 641, 640], 32, 32, 128),    # one query head per kv head
    ([2000, 600, 17, 641, 640], 32, 32, 128),
    ([641, 5, 1300, 639], 4, 4, 64)])
def test_attn_decode_batch_invariant(lens, nh, nkv, d):
    """A sequence's output has the same bits alone and inside a ragged batch."""
    torch = G.torch()
    hs = _hs()
    q, pool, table, _, _ = _paged_case(lens, nh, nkv, d, 77)
    dq = G.to_dev_bf16(q)
    dpool = G.to_dev_bf16(pool.reshape(-1))
    dtab = torch.from_numpy(table).cuda()
    dctx = torch.tensor(lens, dtype=torch.int32).cuda()
    out = torch.zeros((len(lens), nh * d), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_attn_decode(dq.data_ptr(), nh * d, dpool.data_ptr(), dtab.data_ptr(), dctx.data_ptr(),
                        out.data_ptr(), nh * d, len(lens), nh, nkv, d, table.shape[1], max(lens),
                        G.stream_ptr())
    one = torch.zeros((1, nh * d), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_attn_decode(dq.data_ptr(), nh * d, dpool.data_ptr(), dtab.data_ptr(), dctx.data_ptr(),
                        one.data_ptr(), nh * d, 1, nh, nkv, d, table.shape[1], lens[0],
                        G.stream_ptr())
    torch.cuda.synchronize()
    assert np.array_equal(G.from_dev_bf16(one)[0], G.from_dev_bf16(out)[0])


@pytest.mark.parametrize("lens,nh,nkv,d", [
    ([1], 4, 4, 64), ([17, 300, 64, 65], 4, 4, 64), ([5, 130, 1100, 64, 2100], 32, 8, 128),
    ([512], 32, 32, 128), ([2, 129, 700], 8, 2, 128), ([1000, 33], 16, 4, 64),
    ([300, 17, 129], 8, 4, 128),    # two query heads per kv head
    ([700, 641, 640, 1, 129], 8, 8, 128), ([1300, 639, 5, 641], 4, 4, 64)])
def test_attn_decode(lens, nh, nkv, d):
    """One query per sequence (at position ctx - 1) over a paged cache, against
    the oracle's attention; a second call gives the same bits."""
    torch = G.torch()
    hs = _hs()
    q, pool, table, ks, vs = _paged_case(lens, nh, nkv, d, sum(lens) + nh)
    dq = G.to_dev_bf16(q)
    dpool = G.to_dev_bf16(pool.reshape(-1))
    dtab = torch.from_numpy(table).cuda()
    dctx = torch.tensor(lens, dtype=torch.int32).cuda()
    outs = []
    for _ in range(2):
        out = torch.zeros((len(lens), nh * d), dtype=torch.bfloat16, device="cuda")
        hs.hs_k_attn_decode(dq.data_ptr(), nh * d, dpool.data_ptr(), dtab.data_ptr(),
                            dctx.data_ptr(), out.data_ptr(), nh * d, len(lens), nh, nkv, d,
                            table.shape[1], max(lens), G.stream_ptr())
        torch.cuda.synchronize()
        outs.append(G.from_dev_bf16(out))
    assert np.array_equal(outs[0], outs[1])
    for i, n in enumerate(lens):
        ref = attention(q[i].reshape(1, nh, d).astype(np.float64), ks[i].astype(np.float64),
                        vs[i].astype(np.float64), [n - 1], np.arange(n))[0]
        err = np.abs(outs[0][i] - ref).max()
        assert err <= 2e-2 * np.abs(ref).max() + 1e-3, (i, err)


@pytest.mark.parametrize("lens,nh,nkv,d", [
    ([1], 4, 4, 64), ([17, 300, 64, 65], 4, 4, 64), ([5, 130, 1100, 64, 2100], 32, 8, 128),
    ([512], 32, 32, 128), ([1000, 33, 16], 16, 4, 64), ([80, 64, 63, 2], 8, 2, 128),
    ([300, 17, 129], 8, 4, 128), ([650, 640, 3, 576], 8, 8, 128), ([641, 600, 64], 4, 4, 64)])
def test_attn_decode_rope(lens, nh, nkv, d):
    """Decode attention with the step's RoPE and cache append folded in. The
    last position of each sequence is the new token, given before RoPE in a
    QKV row (its pool slot holds garbage that must not be read); against the
    oracle's RoPE and attention, and the appended slot against the rotated
    key (one bf16 rounding) and the value (bitwise)."""
    torch = G.torch()
    hs = _hs()
    q0, pool, table, ks, vs = _paged_case(lens, nh, nkv, d, sum(lens) + 7 * nh)
    rng = np.random.default_rng(len(lens) * 31 + d)
    B, ldqkv, max_ctx = len(lens), (nh + 2 * nkv) * d, max(lens)
    qkv = gen.round_to_bf16((rng.standard_normal((B, ldqkv)) * 1.5).astype(np.float32))
    for i, n in enumerate(lens):
        pool[table[i, (n - 1) // 16], :, :, (n - 1) % 16] = 4096.0
    cos, sin = rope_angles(np.arange(max_ctx), d, 10000.0)
    dcos = torch.from_numpy(np.ascontiguousarray(cos.astype(np.float32))).cuda()
    dsin = torch.from_numpy(np.ascontiguousarray(sin.astype(np.float32))).cuda()
    dqkv = G.to_dev_bf16(qkv)
    dpool = G.to_dev_bf16(pool.reshape(-1))
    dtab = torch.from_numpy(table).cuda()
    dctx = torch.tensor(lens, dtype=torch.int32).cuda()
    out = torch.zeros((B, nh * d), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_attn_decode_rope(dqkv.data_ptr(), ldqkv, dpool.data_ptr(), dtab.data_ptr(),
                             dctx.data_ptr(), dcos.data_ptr(), dsin.data_ptr(), max_ctx,
                             out.data_ptr(), nh * d, B, nh, nkv, d, table.shape[1], max_ctx,
                             G.stream_ptr())
    torch.cuda.synchronize()
    got = G.from_dev_bf16(out)
    pool_after = G.from_dev_bf16(dpool).reshape(pool.shape)
    pool_bits = gen.to_bf16_bits(pool_after)
    for i, n in enumerate(lens):
        c, s_ = cos[n - 1:n], sin[n - 1:n]
        qr = apply_rope(qkv[i, :nh * d].reshape(1, nh, d).astype(np.float64), c, s_)
        kr = apply_rope(qkv[i, nh * d:(nh + nkv) * d].reshape(1, nkv, d).astype(np.float64), c, s_)
        v_new = qkv[i, (nh + nkv) * d:].reshape(1, nkv, d)
        blk, off = table[i, (n - 1) // 16], (n - 1) % 16
        k_slot = pool_after[blk, 0, :, off]
        assert np.abs(k_slot - kr[0]).max() <= 8e-3 * np.abs(kr).max(), i
        assert np.array_equal(pool_bits[blk, 1, :, off], gen.to_bf16_bits(v_new[0])), i
        K = np.concatenate([ks[i][:n - 1], k_slot[None]]).astype(np.float64)
        V = np.concatenate([vs[i][:n - 1], v_new]).astype(np.float64)
        ref = attention(qr, K, V, [n - 1], np.arange(n))[0]
        err = np.abs(got[i] - ref).max()
        assert err <= 2e-2 * np.abs(ref).max() + 1e-3, (i, err)
    # the cached tokens before the new one are untouched
    keep = np.ones(pool.shape[:1] + pool.shape[3:4], bool)
    for i, n in enumerate(lens):
        keep[table[i, (n - 1) // 16], (n - 1) % 16] = False
    before = gen.to_bf16_bits(pool.transpose(0, 3, 1, 2, 4))[keep]
    after = pool_bits.transpose(0, 3, 1, 2, 4)[keep]
    assert np.array_equal(before, after)


def test_attn_decode_rope_rejects_short_tables():
    torch = G.torch()
    hs = _hs()
    buf = torch.zeros(1 << 16, dtype=torch.int32, device="cuda")
    p = buf.data_ptr()
    with pytest.raises(hs.HSError) as e:      # max_pos < max_ctx
        hs.hs_k_attn_decode_rope(p, 384, p, p, p, p, p, 16, p, 128, 1, 1, 1, 128, 2, 32)
    assert e.value.code == hs.HS_EINVAL
    with pytest.raises(hs.HSError) as e:      # QKV rows narrower than the heads
        hs.hs_k_attn_decode_rope(p, 256, p, p, p, p, p, 32, p, 128, 1, 1, 1, 128, 2, 32)
    assert e.value.code == hs.HS_EINVAL


@pytest.mark.parametrize("rows,hidden", [(1, 256), (37, 4096), (5, 5120), (3, 8192)])
def test_rmsnorm(rows, hidden):
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(rows + hidden)
    x = gen.round_to_bf16((rng.standard_normal((rows, hidden)) * 3).astype(np.float32))
    g = gen.round_to_bf16(rng.standard_normal(hidden).astype(np.float32))
    dx, dg = G.to_dev_bf16(x), G.to_dev_bf16(g)
    out = torch.zeros((rows, hidden), dtype=torch.bfloat16, device="cuda")
    hs.hs_k_rmsnorm(dx.data_ptr(), dg.data_ptr(), out.data_ptr(), rows, hidden, 1e-5,
                    G.stream_ptr())
    torch.cuda.synchronize()
    ref = rms_norm(x.astype(np.float64), g.astype(np.float64), 1e-5)
    assert np.max(np.abs(G.from_dev_bf16(out) - ref)) <= 8e-3 * np.abs(ref).max()


# Decode projections with the RMSNorm folded in, one shape per skinny
# variant the stage reaches (7B QKV and gate/up at 1, 8, 12 and 16 tokens)
# plus small ragged ones; rows carry different scales so that a wrong
# per-row 1/RMS shows.
@pytest.mark.parametrize("M,N,K,epi", [
    (1, 12288, 4096, "store"), (8, 22016, 4096, "swiglu"), (16, 28672, 4096, "swiglu"),
    (12, 6144, 4096, "store"), (16, 12288, 4096, "store"), (5, 1536, 256, "resid"),
    (3, 512, 64, "f32"), (16, 1376, 320, "swiglu")])
def test_gemm_rmsnorm(M, N, K, epi):
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(M * 13 + N + K)
    scale = 10.0 ** (np.arange(M) % 3 - 1)[:, None]
    X = gen.round_to_bf16((rng.standard_normal((M, K)) * scale).astype(np.float32))
    g = gen.round_to_bf16((1 + 0.3 * rng.standard_normal(K)).astype(np.float32))
    Wt = gen.round_to_bf16((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
    u = rms_norm(X.astype(np.float64), g.astype(np.float64), 1e-5)
    acc = u @ Wt.astype(np.float64).T
    ncol = N // 2 if epi == "swiglu" else N
    R = gen.round_to_bf16(rng.standard_normal((M, ncol)).astype(np.float32))
    if epi == "swiglu":
        idx = np.arange(ncol)
        ref = silu(acc[:, (idx // 16) * 32 + idx % 16]) * acc[:, (idx // 16) * 32 + 16 + idx % 16]
    elif epi == "resid":
        ref = R + acc
    else:
        ref = acc
    dX, dg = G.to_dev_bf16(X), G.to_dev_bf16(g)
    dW = torch.from_numpy(G.tile_bits(gen.to_bf16_bits(Wt)).view(np.int16)).cuda()
    outs = []
    for _ in range(2):
        if epi == "f32":
            Y = torch.zeros((M, N), dtype=torch.float32, device="cuda")
        elif epi == "resid":
            Y = G.to_dev_bf16(R)
        else:
            Y = torch.zeros((M, ncol), dtype=torch.bfloat16, device="cuda")
        hs.hs_k_gemm_rmsnorm(dX.data_ptr(), K, dg.data_ptr(), 1e-5, dW.data_ptr(), Y.data_ptr(),
                             ncol, Y.data_ptr() if epi == "resid" else 0, ncol, M, N, K, epi,
                             G.stream_ptr())
        torch.cuda.synchronize()
        outs.append(Y.cpu().numpy() if epi == "f32" else G.from_dev_bf16(Y))
    assert np.array_equal(outs[0], outs[1])
    # per row: the bf16 rounding of the normalised activations dominates
    for m in range(M):
        err = np.abs(outs[0][m] - ref[m]).max()
        assert err <= 8e-3 * np.abs(ref[m]).max() + 1e-6, (m, err)
    # the fused norm does not depend on the other rows of the batch
    if M > 1:
        Y1 = torch.zeros((1, N), dtype=torch.float32, device="cuda") if epi == "f32" else (
            G.to_dev_bf16(R[-1:]) if epi == "resid" else
            torch.zeros((1, ncol), dtype=torch.bfloat16, device="cuda"))
        hs.hs_k_gemm_rmsnorm(dX[-1:].data_ptr(), K, dg.data_ptr(), 1e-5, dW.data_ptr(),
                             Y1.data_ptr(), ncol, Y1.data_ptr() if epi == "resid" else 0, ncol,
                             1, N, K, epi, G.stream_ptr())
        torch.cuda.synchronize()
        last = Y1.cpu().numpy() if epi == "f32" else G.from_dev_bf16(Y1)
        assert np.array_equal(last[0], outs[0][-1])


def test_gemm_rmsnorm_rejects_unsupported_shapes():
    torch = G.torch()
    hs = _hs()
    buf = torch.zeros(1 << 16, dtype=torch.bfloat16, device="cuda")
    p = buf.data_ptr()
    for (M, N, K) in ((17, 64, 64), (0, 64, 64), (4, 64, 72)):
        with pytest.raises(hs.HSError) as e:
            hs.hs_k_gemm_rmsnorm(p, 128, p, 1e-5, p, p, N, 0, 0, M, N, K, 0)
        assert e.value.code == hs.HS_EINVAL


def test_gemm_rejects_unsupported_shapes():
    torch = G.torch()
    hs = _hs()
    buf = torch.zeros(1 << 16, dtype=torch.bfloat16, device="cuda")
    p = buf.data_ptr()
    for (M, N, K, epi, ldx) in ((8, 24, 64, 0, 64), (8, 64, 12, 0, 64), (8, 48, 64, 2, 64),
                                (0, 64, 64, 0, 64), (8, 64, 72, 0, 72)):
        with pytest.raises(hs.HSError) as e:
            hs.hs_k_gemm(p, ldx, p, p, N, 0, 0, M, N, K, epi)
        assert e.value.code == hs.HS_EINVAL


@pytest.mark.parametrize("n_rows,n_cols", [(1, 4), (3, 1024), (2, 4096), (5, 32000),
                                            (2, 128256), (1, 8196)])
def test_argmax_ties_lowest_index(n_rows, n_cols):
    """Greedy sampling: the lowest index of the row maximum, with ties inside a
    4096-column chunk, across a chunk boundary (the earlier chunk must win)
    and at the last column; the rows are checked against numpy's argmax,
    which returns the first maximal index."""
    torch = G.torch()
    hs = _hs()
    rng = np.random.default_rng(n_rows * 31 + n_cols)
    x = rng.standard_normal((n_rows, n_cols)).astype(np.float32)
    top = np.float32(50.0)
    for r in range(n_rows):
        kind = r % 5
        if kind == 0:      # tie inside one chunk
            cols = rng.choice(min(n_cols, 4096), size=min(3, n_cols), replace=False)
        elif kind == 1:    # tie across the chunk boundary and at the last column
            cols = [c for c in (4095, 4096, n_cols - 1) if c < n_cols]
        elif kind == 2:    # maximum only at the last column
            cols = [n_cols - 1]
        elif kind == 3:    # every column equal
            x[r, :] = top
            cols = []
        else:              # ties in the last chunk and the first
            cols = sorted({n_cols - 1, n_cols - 2, 0} & set(range(n_cols)))
        x[r, list(cols)] = top
    x[0, -1] = np.inf if n_cols > 8 and n_rows > 2 else x[0, -1]
    dx = torch.from_numpy(x).cuda()
    out = torch.full((n_rows,), -1, dtype=torch.int32, device="cuda")
    hs.hs_k_argmax(dx.data_ptr(), n_rows, n_cols, out.data_ptr(), G.stream_ptr())
    torch.cuda.synchronize()
    assert out.cpu().numpy().tolist() == np.argmax(x, axis=1).tolist()


def test_argmax_rejects_bad_shapes():
    torch = G.torch()
    hs = _hs()
    x = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    out = torch.zeros(2, dtype=torch.int32, device="cuda")
    for rows, cols in [(0, 8), (2, 0), (2, 6)]:
        with pytest.raises(hs.HSError) as e:
            hs.hs_k_argmax(x.data_ptr(), rows, cols, out.data_ptr(), G.stream_ptr())
        assert e.value.code == hs.HS_EINVAL
