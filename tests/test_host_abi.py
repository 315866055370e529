"""Host-side checks of libhs.so that need no GPU: exported symbols, weight
layout, image packing, blob header codec and argument validation."""
import os
import re

import numpy as np
import pytest

import oracle
from oracle import kvblob
from workloads import MODELS, gen
from paper_2502_15524_amd import hs, pipeline
from tests.gpu_util import tile_bits, untile_bits

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header):
    with open(os.path.join(ROOT, "include", header)) as f:
        src = f.read()
    return set(re.findall(r"^\s*(?:hs_status|const char\*)\s+(hs_\w+)\s*\(", src, re.M))


def test_library_exports_every_declared_symbol():
    lib = hs.lib()
    declared = _declared("hs.h") | _declared("hs_kernel.h")
    assert {"hs_stage_create", "hs_stage_load_chunk", "hs_stage_prefill", "hs_stage_decode",
            "hs_kv_export", "hs_kv_import", "hs_stage_merge"} <= declared
    for name in declared:
        assert hasattr(lib, name), name
    assert set(hs.EXPORTED) == declared


@pytest.mark.parametrize("name", ["llama2-7b", "llama2-13b", "llama3-8b", "tiny"])
def test_layout_matches_parameter_accounting(name):
    cfg = MODELS[name]
    c = pipeline.hs_cfg(cfg)
    descs, nbytes = hs.hs_weight_layout(c, 0, cfg.n_layers)
    # tiled matrices pad their input dimension to a multiple of 64 (only the
    # tiny model's FFN width 688 is not one)
    pad = 0 if cfg.ffn % 64 == 0 else cfg.n_layers * cfg.hidden * (-cfg.ffn % 64) * 2
    assert nbytes == oracle.image_bytes_16bit(cfg) + pad
    assert sum(d["bytes"] for d in descs) == oracle.image_bytes_16bit(cfg) + pad
    prev_end = 0
    for d in descs:
        assert d["offset"] % 256 == 0 and d["offset"] >= prev_end
        kp = -(-d["cols"] // 64) * 64 if d["tiled"] else d["cols"]
        assert d["bytes"] == d["rows"] * kp * 2
        assert d["tiled"] == (d["kind"] in (hs.HS_W_QKV, hs.HS_W_O, hs.HS_W_GATEUP,
                                            hs.HS_W_DOWN, hs.HS_W_LM_HEAD))
        prev_end = d["offset"] + d["bytes"]
    # stage cuts
    per = cfg.n_layers // 4 if cfg.n_layers % 4 == 0 else cfg.n_layers
    for b in range(0, cfg.n_layers, per):
        _, sb = hs.hs_weight_layout(c, b, b + per)
        assert sb == oracle.image_bytes_16bit(cfg, b, b + per) + pad * per // cfg.n_layers


def test_seven_b_middle_stage_image_bytes():
    cfg = MODELS["llama2-7b"]
    _, nb = hs.hs_weight_layout(pipeline.hs_cfg(cfg), 8, 16)
    assert nb == 3_238_133_760


def test_layers_are_contiguous_byte_ranges():
    cfg = MODELS["tiny"]
    descs, _ = hs.hs_weight_layout(pipeline.hs_cfg(cfg), 0, 2)
    for l in range(2):
        ds = [d for d in descs if d["layer"] == l]
        assert [d["kind"] for d in ds] == [hs.HS_W_ATTN_NORM, hs.HS_W_QKV, hs.HS_W_O,
                                           hs.HS_W_FFN_NORM, hs.HS_W_GATEUP, hs.HS_W_DOWN]
        for a, b in zip(ds, ds[1:]):
            assert b["offset"] - (a["offset"] + a["bytes"]) < 256


def test_image_put_places_tensors():
    cfg = MODELS["tiny"]
    c = pipeline.hs_cfg(cfg)
    descs, nb = hs.hs_weight_layout(c, 1, 2)
    img = np.zeros(nb, np.uint8)
    pipeline.pack_image(cfg, 1, 2, img.ctypes.data)
    by_kind = {d["kind"]: d for d in descs}
    u16 = img.view(np.uint16)

    def tensor(kind):
        d = by_kind[kind]
        raw = u16[d["offset"] // 2:(d["offset"] + d["bytes"]) // 2]
        if d["tiled"]:
            return untile_bits(raw, d["rows"], d["cols"])
        return raw.reshape(d["rows"], d["cols"])

    qkv = tensor(hs.HS_W_QKV)
    wq = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wq"))
    wk = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wk"))
    wv = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wv"))
    # q and k heads (d = 64): rows 16j + r of the first half at 32j + r, their
    # RoPE partners (row + 32) at 32j + 16 + r; v rows in order
    d = cfg.head_dim
    for h in range(cfg.n_heads):
        for i in range(d):
            j, r, second = (i % (d // 2)) // 16, i % 16, i // (d // 2)
            stored = h * d + 32 * j + 16 * second + r
            assert np.array_equal(qkv[stored], wq[h * d + i])
            assert np.array_equal(qkv[256 + stored], wk[h * d + i])
    assert np.array_equal(qkv[512:], wv)
    gu = tensor(hs.HS_W_GATEUP)
    g = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wgate"))
    u = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wup"))
    for f in (0, 15, 16, 100, 687):
        assert np.array_equal(gu[(f // 16) * 32 + f % 16], g[f])
        assert np.array_equal(gu[(f // 16) * 32 + 16 + f % 16], u[f])
    assert np.all(tensor(hs.HS_W_ATTN_NORM) == 0x3F80)   # bf16 1.0
    d = by_kind[hs.HS_W_DOWN]                             # 688 columns padded to 704
    raw = u16[d["offset"] // 2:(d["offset"] + d["bytes"]) // 2]
    wd = gen.to_bf16_bits(gen.weight_f32(cfg, 1, "wdown"))
    assert np.array_equal(raw, tile_bits(wd))
    with pytest.raises(hs.HSError) as e:
        hs.hs_image_put(c, 1, 2, 0, "wq", wq.ctypes.data, wq.size, img.ctypes.data)
    assert e.value.code == hs.HS_EINVAL
    with pytest.raises(hs.HSError):
        hs.hs_image_put(c, 1, 2, 1, "wq", wq.ctypes.data, wq.size - 1, img.ctypes.data)
    with pytest.raises(hs.HSError):
        hs.hs_image_put(c, 1, 2, -1, "embed", wq.ctypes.data, wq.size, img.ctypes.data)


def _oracle_blob():
    rng = np.random.default_rng(9)
    seqs = []
    for sid, n in ((5, 3), (1 << 40, 33)):
        seqs.append((sid, rng.integers(0, 65536, (2, n, 4, 64), dtype=np.uint16),
                     rng.integers(0, 65536, (2, n, 4, 64), dtype=np.uint16)))
    return kvblob.pack(3, 5, 4, 64, 16, seqs)


def test_blob_header_codec_agrees_with_oracle_codec():
    blob = _oracle_blob()
    info = hs.hs_kv_blob_describe(blob[:64 + 32])
    assert info["layer_begin"] == 3 and info["layer_end"] == 5
    assert info["n_kv_heads"] == 4 and info["head_dim"] == 64 and info["block_size"] == 16
    assert info["n_seqs"] == 2 and info["total_bytes"] == len(blob)
    assert info["payload_offset"] == 256
    assert info["payload_bytes"] == 2 * (1 + 3) * 2 * 4 * 16 * 64 * 2


@pytest.mark.parametrize("mutate", ["magic", "version", "truncated", "blocks", "size", "dup"])
def test_blob_header_rejects_corruption(mutate):
    blob = bytearray(_oracle_blob())
    if mutate == "magic":
        blob[0:4] = b"XXXX"
    elif mutate == "version":
        blob[4] = 2
    elif mutate == "truncated":
        blob = blob[:70]
    elif mutate == "blocks":
        blob[76] = 9           # n_blocks of the first record
    elif mutate == "size":
        blob[56] ^= 1          # total_bytes
    elif mutate == "dup":
        blob[80:88] = blob[64:72]  # second record gets the first id
    with pytest.raises(hs.HSError) as e:
        hs.hs_kv_blob_describe(bytes(blob[:64 + 32]) if mutate != "truncated" else bytes(blob))
    assert e.value.code == hs.HS_EINVAL


def test_stage_create_validates_before_touching_the_gpu():
    c = pipeline.hs_cfg(MODELS["tiny"])
    for opts, rng in ((hs.stage_opts(1, 64, 64, kv_block_size=8), (0, 2)),
                      (hs.stage_opts(0, 64, 64), (0, 2)),
                      (hs.stage_opts(1, 64, 64, n_copy_streams=0), (0, 2)),
                      (hs.stage_opts(1, 64, 64), (1, 3)),
                      (hs.stage_opts(1, 64, 64, resident=(1, 2)), (0, 2))):
        with pytest.raises(hs.HSError) as e:
            hs.hs_stage_create(c, rng[0], rng[1], opts)
        assert e.value.code == hs.HS_EINVAL
    bad = pipeline.hs_cfg(MODELS["tiny"])
    bad.head_dim = 96
    with pytest.raises(hs.HSError) as e:
        hs.hs_weight_layout(bad, 0, 2)
    assert e.value.code == hs.HS_EINVAL


def test_tiled_pack_matches_format_description():
    """The library's packer agrees with the tiled format as documented."""
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 65536, (24, 200), dtype=np.uint16)
    dst = np.zeros(24 * 256, np.uint16)
    hs.hs_pack_tiled(bits.ctypes.data, 24, 200, dst.ctypes.data)
    assert np.array_equal(dst, tile_bits(bits))
    # one element by hand: row 10, column 75 -> block (kb 1, nb 1), row 2, chunk 1
    off = ((1 * 3 + 1) * 1024 + 2 * 128 + ((1 ^ 2) * 16) + 3 * 2) // 2
    assert dst[off] == bits[10, 75]
    assert np.all(untile_bits(dst, 24, 256)[:, 200:] == 0)
    with pytest.raises(hs.HSError):
        hs.hs_pack_tiled(bits.ctypes.data, 20, 200, dst.ctypes.data)
