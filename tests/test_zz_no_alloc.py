"""hs_k_attn_decode_noalloc: the decode attention with its split partials in
the library's static per-GPU array. Its results must be those of
hs_k_attn_decode bit for bit (same kernels, same split order), on calls in
a row that reuse the array, the second smaller than the first; sizes beyond
the array are refused before the GPU is touched."""
import numpy as np
import pytest

from oracle.llama import attention
from tests import gpu_util as G
from tests.test_gpu_kernels import _paged_case


def _hs():
    from paper_2502_15524_amd import hs
    return hs


def test_noalloc_rejects_sizes_beyond_the_static_array():
    """Runs without a GPU: the size check precedes every HIP call."""
    hs = _hs()
    p = 1 << 20   # any non-null value: nothing is dereferenced or launched
    # 64 sequences x 64 heads x 64 splits (8192 tokens) x 130 floats = 34 M > 8 M floats
    with pytest.raises(hs.HSError) as e:
        hs.hs_k_attn_decode_noalloc(p, 64 * 128, p, p, p, p, 64 * 128, 64, 64, 8, 128, 512,
                                    8192)
    assert e.value.code == hs.HS_ERANGE
    with pytest.raises(hs.HSError) as e:    # argument errors as hs_k_attn_decode
        hs.hs_k_attn_decode_noalloc(p, 128, p, p, p, p, 128, 1, 3, 2, 128, 4, 64)
    assert e.value.code == hs.HS_EINVAL


def _run(fn, case, lens, nh, nkv, d):
    torch = G.torch()
    q, pool, table, _, _ = case
    dq = G.to_dev_bf16(q)
    dpool = G.to_dev_bf16(pool.reshape(-1))
    dtab = torch.from_numpy(table).cuda()
    dctx = torch.tensor(lens, dtype=torch.int32).cuda()
    out = torch.full((len(lens), nh * d), float("nan"), dtype=torch.bfloat16, device="cuda")
    fn(dq.data_ptr(), nh * d, dpool.data_ptr(), dtab.data_ptr(), dctx.data_ptr(), out.data_ptr(),
       nh * d, len(lens), nh, nkv, d, table.shape[1], max(lens), G.stream_ptr())
    torch.cuda.synchronize()
    return G.from_dev_bf16(out)


@pytest.mark.gpu
def test_noalloc_matches_allocating_entry_on_two_calls():
    """Two calls in a row through the C ABI, the second with fewer sequences,
    heads and tokens than the first (so the array still holds the first
    call's partials past what the second writes): each equals
    hs_k_attn_decode bitwise, and the oracle's attention within the kernel
    tolerance."""
    hs = _hs()
    cases = [([2100, 5, 1300, 129, 700, 2048, 17, 1900], 32, 8, 128, 11),
             ([300, 64, 1], 4, 4, 64, 12)]
    for lens, nh, nkv, d, seed in cases:
        print(f"[noalloc] lens={lens} heads={nh}/{nkv} d={d}", flush=True)
        case = _paged_case(lens, nh, nkv, d, seed)
        got = _run(hs.hs_k_attn_decode_noalloc, case, lens, nh, nkv, d)
        ref = _run(hs.hs_k_attn_decode, case, lens, nh, nkv, d)
        assert np.array_equal(got, ref)
        q, _, _, ks, vs = case
        for i, n in enumerate(lens):
            o = attention(q[i].reshape(1, nh, d).astype(np.float64), ks[i].astype(np.float64),
                          vs[i].astype(np.float64), [n - 1], np.arange(n))[0]
            assert np.abs(got[i] - o).max() <= 2e-2 * np.abs(o).max() + 1e-3, i
