"""The C-ABI library loads, exports every entry point of include/sats.h, and
rejects bad arguments before touching the GPU (no device needed)."""
import ctypes
import os
import re

import pytest

import paper_2607_08991_amd as sats
from paper_2607_08991_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sats.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sats_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    syms = declared_symbols()
    for name in ["sats_mlp_forward", "sats_mlp_dense", "sats_mlp_forward_f32", "sats_mlp_dense_f32",
                 "sats_mlp_forward_inspect", "sats_last_error"]:
        assert name in syms


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    missing = [s for s in declared_symbols() if not hasattr(lib, s)]
    assert not missing, missing
    assert set(declared_symbols()) == set(_lib.SIGNATURES)


def test_library_is_built_for_gfx950():
    data = open(_lib.LIB_PATH, "rb").read()
    assert b"gfx950" in data


FAKE = 1 << 20  # a non-null address: never dereferenced by the host checks below


def fwd(**kw):
    args = dict(x=FAKE, ids=FAKE, wg=FAKE, wu=FAKE, wd=FAKE, thr=FAKE, lut=FAKE, out=FAKE * 16,
                n=1, d=8, dff=8, L=1)
    args.update(kw)
    a = args
    return sats.load().sats_mlp_forward(a["x"], a["ids"], a["wg"], a["wu"], a["wd"], a["thr"],
                                        a["lut"], a["out"], a["n"], a["d"], a["dff"], a["L"], None)


@pytest.mark.parametrize("field", ["x", "wg", "wu", "wd", "out", "thr"])
def test_null_pointers_rejected(field):
    assert fwd(**{field: None}) == _lib.SATS_ERR_NULL
    assert sats.sats_last_error()


def test_ids_required_with_lut_but_not_without():
    assert fwd(ids=None) == _lib.SATS_ERR_NULL
    assert "token_ids" in sats.sats_last_error()
    assert fwd(ids=None, lut=None, n=0) == _lib.SATS_OK


@pytest.mark.parametrize("kw", [dict(d=0), dict(dff=0), dict(L=0), dict(n=-1), dict(d=1 << 25)])
def test_bad_shapes_rejected(kw):
    assert fwd(**kw) == _lib.SATS_ERR_SHAPE


def test_zero_tokens_is_a_no_op():
    assert fwd(n=0) == _lib.SATS_OK
    assert sats.sats_last_error() == ""
    lib = sats.load()
    assert lib.sats_mlp_dense(FAKE, FAKE, FAKE, FAKE, FAKE, 0, 8, 8, 1, None) == _lib.SATS_OK


def test_partial_overlap_of_out_and_x_rejected():
    # x spans [FAKE, FAKE + 2*8*2) in bf16; out starting 2 bytes in overlaps without being equal
    assert fwd(n=2, out=FAKE + 2) == _lib.SATS_ERR_ARG
    assert "overlap" in sats.sats_last_error()


def test_dense_needs_no_thresholds_but_checks_weights():
    lib = sats.load()
    assert lib.sats_mlp_dense(FAKE, None, FAKE, FAKE, FAKE, 1, 8, 8, 1, None) == _lib.SATS_ERR_NULL


def test_reserve_rejects_bad_element_size():
    assert sats.load().sats_reserve(4, 8, 8, 1, 3, None) == _lib.SATS_ERR_ARG


def fwd_lora(rank=16, scale=0.5, **kw):
    ad = dict(ag=FAKE, bg=FAKE, au=FAKE, bu=FAKE, adn=FAKE, bd=FAKE)
    ad.update({k: kw.pop(k) for k in list(kw) if k in ad})
    a = dict(x=FAKE, ids=FAKE, wg=FAKE, wu=FAKE, wd=FAKE, thr=FAKE, lut=FAKE, out=FAKE * 16, n=1, d=8, dff=8, L=1)
    a.update(kw)
    return sats.load().sats_mlp_forward_lora(a["x"], a["ids"], a["wg"], a["wu"], a["wd"], ad["ag"], ad["bg"],
                                             ad["au"], ad["bu"], ad["adn"], ad["bd"], rank, scale, a["thr"],
                                             a["lut"], a["out"], a["n"], a["d"], a["dff"], a["L"], None, None,
                                             None, None, None)


@pytest.mark.parametrize("field", ["ag", "bg", "au", "bu", "adn", "bd"])
def test_lora_needs_every_adapter(field):
    assert fwd_lora(**{field: None}) == _lib.SATS_ERR_NULL
    assert "adapter" in sats.sats_last_error()


@pytest.mark.parametrize("rank", [0, 4, 12, 128])
def test_lora_rank_rejected(rank):
    assert fwd_lora(rank=rank) == _lib.SATS_ERR_SHAPE
    assert "rank" in sats.sats_last_error()


def test_lora_alignment_and_scale_rejected():
    assert fwd_lora(bd=FAKE + 2) == _lib.SATS_ERR_ARG
    assert fwd_lora(scale=float("nan")) == _lib.SATS_ERR_ARG
    assert fwd_lora(rank=12, n=0) == _lib.SATS_OK  # zero tokens: nothing to do


def test_route_table_arguments_rejected():
    lib = sats.load()

    def call(table=FAKE, n=10, nh=10, vocab=100, r_tar=0.5, ids=FAKE):
        return lib.sats_route_table(FAKE, FAKE, ids, n, FAKE, nh, vocab, r_tar, table, None, None, None, None)
    assert call(table=None) == _lib.SATS_ERR_NULL
    assert call(ids=None) == _lib.SATS_ERR_NULL
    assert call(vocab=0) == _lib.SATS_ERR_SHAPE
    assert call(n=-1) == _lib.SATS_ERR_SHAPE
    assert call(r_tar=1.5) == _lib.SATS_ERR_ARG
    assert call(r_tar=float("nan")) == _lib.SATS_ERR_ARG


def test_timing_kinds_match_the_header_and_name_their_kernels():
    text = open(HEADER).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"\b(SATS_K_[A-Z_]+)\s*=\s*(\d+)", text))
    count = enum.pop("SATS_K_COUNT")
    assert sorted(enum.values()) == list(range(count))
    for name, value in enum.items():
        assert getattr(sats, name) == value, name
        kernel = sats.sats_kernel_name(value)
        assert "kernel" in kernel, (name, kernel)
    assert sats.sats_kernel_name(sats.SATS_K_LORA_V) == "lora_v_kernel"
    with pytest.raises(sats.SatsError):
        sats.sats_timing_begin(count, 1)


# ------------------------------------------------------------------ options and path selection

def test_options_are_validated_and_reset():
    lib = sats.load()
    for bad in (dict(batch_path=4), dict(batch_path=-1), dict(single_token=2), dict(dec_block_cols=-1),
                dict(dec_block_cols=65), dict(lora_per_token=2)):
        o = _lib.SatsOptions(**{**dict(batch_path=0, single_token=0, dec_block_cols=0, lora_per_token=0), **bad})
        assert lib.sats_set_options(ctypes.byref(o)) == _lib.SATS_ERR_ARG, bad
    assert lib.sats_set_options(None) == _lib.SATS_OK


def test_query_path_follows_shapes_and_options():
    q = sats.sats_query_path
    L8B = (4096, 14336)
    assert q(0, *L8B, 2, n_cus=256) == 0
    assert q(1, *L8B, 2, n_cus=256) == sats.SATS_PATH_SINGLE_TOKEN
    assert q(1, *L8B, 4, n_cus=256) == sats.SATS_PATH_SINGLE_TOKEN
    assert q(4, *L8B, 2, n_cus=256) == sats.SATS_PATH_BATCH_MFMA
    assert q(4, *L8B, 4, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT       # fp32 batches: compacted kernels
    assert q(1, *L8B, 2, aligned16=False, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT
    assert q(1, 5000, 64, 2, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT    # h does not fit the LDS copy
    with sats.options(batch_path=sats.SATS_BATCH_SPLIT, single_token=sats.SATS_SINGLE_OFF):
        assert q(4, *L8B, 2, n_cus=256) == sats.SATS_PATH_BATCH_SPLIT
        assert q(1, *L8B, 2, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT
    with sats.options(batch_path=sats.SATS_BATCH_COMPACT):
        assert q(4, *L8B, 2, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT
    assert q(4, *L8B, 2, n_cus=256) == sats.SATS_PATH_BATCH_MFMA          # defaults restored


def test_single_token_path_refuses_matrices_of_2gb():
    """The single-token kernels address a matrix with 32-bit buffer offsets
    (0x80000000 reads zeros), so a layer whose matrix reaches 2^31 bytes
    takes the compacted kernels (64-bit indices) instead."""
    q = sats.sats_query_path
    assert q(1, 4096, 131072 - 16, 4, n_cus=256) == sats.SATS_PATH_SINGLE_TOKEN   # just below 2 GB
    assert q(1, 4096, 131072, 4, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT       # exactly 2 GB
    assert q(1, 4096, 262144, 2, n_cus=256) == sats.SATS_PATH_BATCH_COMPACT       # bf16, 2 GB
    assert q(1, 4096, 262144 - 8, 2, n_cus=256) == sats.SATS_PATH_SINGLE_TOKEN


def test_query_path_rejects_bad_arguments():
    lib = sats.load()
    p = ctypes.c_int(0)
    assert lib.sats_query_path(1, 8, 8, 3, 1, 256, ctypes.byref(p)) == _lib.SATS_ERR_ARG
    assert lib.sats_query_path(1, 0, 8, 2, 1, 256, ctypes.byref(p)) == _lib.SATS_ERR_SHAPE
    assert lib.sats_query_path(1, 8, 8, 2, 1, 256, None) == _lib.SATS_ERR_NULL


def test_noalloc_rejects_a_call_past_its_scratch_before_device_work():
    lib = sats.load()
    rc = lib.sats_mlp_forward_noalloc(FAKE, None, FAKE, FAKE, FAKE, FAKE, None, FAKE * 4096, 64, 4096, 14336, 1,
                                      None)
    assert rc == _lib.SATS_ERR_WORKSPACE
    assert "allocation-free" in sats.sats_last_error()
