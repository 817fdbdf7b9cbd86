"""The C ABI library: it loads, exports every function include/cachegen.h declares, and its
host-side validation returns the documented error codes before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2310_07240_amd import cachegen as cg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "cachegen.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(cg_[a-z_0-9]+)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("cg_fit_cdf", "cg_encode", "cg_decode"):
        assert n in names
    assert set(names) == set(cg.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = cg.lib()
    for n in declared_functions():
        assert hasattr(lib, n), n


def P(**kw):
    d = dict(n_ctx=1, n_layers=2, n_tokens=100, n_channels=70, layer_bin=(0.5, 1.0),
             level_mult=(1.0, 2.0), group_size=10, chunk_len=48)
    d.update(kw)
    return cg.CodecParams(**d)


def test_size_queries():
    p = P()
    assert cg.cg_num_chunks(p) == 3
    assert cg.cg_num_streams(p) == 1 * 3 * 2 * 2 * 70
    # per stream: ceil((18 n + 2) / 32) for n = 48, 48, 4 tokens
    per = 2 * 2 * 70
    assert cg.cg_encode_bound_words(p) == per * (2 * ((18 * 48 + 2 + 31) // 32) + (18 * 4 + 2 + 31) // 32) + 8
    assert cg.cg_encode_workspace_bytes(p) > cg.cg_encode_bound_words(p) * 4


@pytest.mark.parametrize("kw", [dict(n_ctx=0), dict(n_layers=0, layer_bin=()), dict(n_tokens=-1),
                                dict(n_channels=0), dict(group_size=0), dict(chunk_len=0),
                                dict(level_mult=()), dict(level_mult=(1.0,) * 9)])
def test_bad_shapes_rejected(kw):
    p = P(**kw)
    assert cg.cg_num_streams(p) == 0
    assert cg.cg_encode_bound_words(p) == 0


@pytest.mark.parametrize("kw", [dict(layer_bin=(0.5, 0.0)), dict(layer_bin=(0.5, float("nan"))),
                                dict(level_mult=(1.0, -2.0)), dict(level_mult=(float("inf"),))])
def test_bad_params_rejected(kw):
    p = P(**kw)
    s, keep = p.c()
    rc = cg.lib().cg_fit_cdf(ctypes.byref(s), ctypes.c_void_p(16), 0, None, ctypes.c_void_p(16), None)
    assert rc == -6


def test_host_validation_before_any_launch():
    """Every error below is decided on the host; no pointer is dereferenced."""
    lib = cg.lib()
    p = P()
    s, keep = p.c()
    fake = ctypes.c_void_p(1 << 20)
    # level out of range, null output
    assert lib.cg_fit_cdf(ctypes.byref(s), fake, 2, None, fake, None) == -1
    assert lib.cg_fit_cdf(ctypes.byref(s), fake, 0, None, None, None) == -1
    # capacity too small
    bound = cg.cg_encode_bound_words(p)
    ws = cg.cg_encode_workspace_bytes(p)
    rc = lib.cg_encode(ctypes.byref(s), fake, fake, fake, fake, fake, bound - 1, fake, fake, fake,
                       ws, None)
    assert rc == -3
    rc = lib.cg_encode(ctypes.byref(s), fake, fake, fake, fake, fake, bound, fake, fake, fake,
                       ws - 1, None)
    assert rc == -3
    # chunk range out of range
    assert lib.cg_decode(ctypes.byref(s), fake, fake, fake, fake, fake, fake, 0, 4, fake, None) == -1
    assert lib.cg_decode(ctypes.byref(s), fake, fake, fake, fake, fake, fake, 2, 1, fake, None) == -1
    # empty range is a no-op
    assert lib.cg_decode(ctypes.byref(s), fake, fake, fake, fake, fake, fake, 1, 1, fake, None) == 0
    # null params
    assert lib.cg_decode(None, fake, fake, fake, fake, fake, fake, 0, 1, fake, None) == -1
    assert cg.strerror(-3).startswith("output or workspace")
    assert cg.strerror(12345) == "unknown error code"


def test_token_layout_size_queries_and_host_validation():
    """Token-parallel layout: one stream per (context, layer, K/V, token), worst case
    ceil((18 C + 2) / 32) words each; capacity errors are decided on the host."""
    lib = cg.lib()
    p = P()
    assert cg.cg_num_token_streams(p) == 1 * 2 * 2 * 100
    per = (18 * 70 + 2 + 31) // 32
    assert cg.cg_encode_tokens_bound_words(p) == 400 * per + 8
    assert cg.cg_decode_tokens_workspace_bytes(p) == 1 * 2 * 2 * 100 * 70
    assert cg.cg_encode_tokens_workspace_bytes(p) > cg.cg_decode_tokens_workspace_bytes(p)
    assert cg.cg_num_token_streams(P(n_channels=0)) == 0
    s, keep = p.c()
    fake = ctypes.c_void_p(1 << 20)
    bound = cg.cg_encode_tokens_bound_words(p)
    ws = cg.cg_encode_tokens_workspace_bytes(p)
    assert lib.cg_encode_tokens(ctypes.byref(s), fake, fake, fake, fake, fake, bound - 1, fake,
                                fake, fake, ws, None) == -3
    assert lib.cg_encode_tokens(ctypes.byref(s), fake, fake, fake, fake, fake, bound, fake, fake,
                                fake, ws - 1, None) == -3
    dws = cg.cg_decode_tokens_workspace_bytes(p)
    assert lib.cg_decode_tokens(ctypes.byref(s), fake, fake, fake, fake, fake, fake, fake, fake,
                                dws - 1, None) == -3
    assert lib.cg_decode_tokens(ctypes.byref(s), fake, fake, fake, fake, fake, fake, None, fake,
                                dws, None) == -1


def test_alignment_is_checked_the_same_way_everywhere():
    """Tables need 16-byte alignment in every call that takes them (the fit writes what the
    decoder later reads with 16-byte loads), scales 4 bytes, offsets 8; decided on the host."""
    lib = cg.lib()
    p = P()
    s, keep = p.c()
    A = 1 << 20
    ok, t8, odd2 = ctypes.c_void_p(A), ctypes.c_void_p(A + 8), ctypes.c_void_p(A + 2)
    # fit: tables 8-byte aligned are rejected (anchor or delta), 16-byte aligned accepted up to
    # the launch (not reached: the level is out of range)
    assert lib.cg_fit_cdf(ctypes.byref(s), ok, 0, t8, ok, None) == -1
    assert lib.cg_fit_cdf(ctypes.byref(s), ok, 0, None, t8, None) == -1
    assert lib.cg_fit_cdf(ctypes.byref(s), ok, 5, ok, ok, None) == -1
    ws = ctypes.c_void_p(A)
    assert lib.cg_fit_cdf_global(ctypes.byref(s), ok, 0, None, t8, ws, 8192, None) == -1
    # encode: misaligned tables
    bound = cg.cg_encode_bound_words(p)
    wsb = cg.cg_encode_workspace_bytes(p)
    assert lib.cg_encode(ctypes.byref(s), ok, ok, t8, ok, ok, bound, ok, ok, ws, wsb, None) == -1
    assert lib.cg_encode(ctypes.byref(s), ok, ok, ok, t8, ok, bound, ok, ok, ws, wsb, None) == -1
    # decode: misaligned scales, tables, offsets
    assert lib.cg_decode(ctypes.byref(s), ok, ok, odd2, ok, ok, ok, 0, 1, ok, None) == -1
    assert lib.cg_decode(ctypes.byref(s), ok, ok, ok, ok, t8, ok, 0, 1, ok, None) == -1
    assert lib.cg_decode(ctypes.byref(s), ok, ctypes.c_void_p(A + 4), ok, ok, ok, ok, 0, 1, ok,
                         None) == -1
    # streamed decode: misaligned device scales
    assert lib.cg_decode_streamed(ctypes.byref(s), ok, ok, ok, 1 << 20, ok, odd2, ok, ok, ok, ok,
                                  0.0, None, None, None) == -1
    # token layout decode: misaligned scales
    dws = cg.cg_decode_tokens_workspace_bytes(p)
    assert lib.cg_decode_tokens(ctypes.byref(s), ok, ok, odd2, ok, ok, ok, ok, ws, dws, None) == -1
    # status: null or misaligned workspace
    assert lib.cg_get_status(None, None) == -1
    assert lib.cg_get_status(ctypes.c_void_p(A + 2), None) == -1
    # all-level fit: misaligned tables, status or scales
    assert lib.cg_fit_cdf_levels(ctypes.byref(s), ok, t8, ok, None, None, None) == -1
    assert lib.cg_fit_cdf_levels(ctypes.byref(s), ok, ok, t8, None, None, None) == -1
    assert lib.cg_fit_cdf_levels(ctypes.byref(s), ok, ok, ok, odd2, None, None) == -1
    assert lib.cg_fit_cdf_levels(ctypes.byref(s), ok, ok, ok, None, odd2, None) == -1
    assert lib.cg_fit_cdf_levels(ctypes.byref(s), ok, None, ok, None, None, None) == -1
    # encode with given scales: misaligned or missing scales, misaligned tables
    assert lib.cg_encode_with_scales(ctypes.byref(s), ok, ok, ok, ok, odd2, ok, bound, ok, ws,
                                     wsb, None) == -1
    assert lib.cg_encode_with_scales(ctypes.byref(s), ok, ok, ok, ok, None, ok, bound, ok, ws,
                                     wsb, None) == -1
    assert lib.cg_encode_with_scales(ctypes.byref(s), ok, ok, t8, ok, ok, ok, bound, ok, ws,
                                     wsb, None) == -1
    assert lib.cg_encode_with_scales(ctypes.byref(s), ok, ok, ok, ok, ok, ok, bound - 1, ok, ws,
                                     wsb, None) == -3
