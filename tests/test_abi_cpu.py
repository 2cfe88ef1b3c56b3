"""CPU-side checks of the C ABI: the library loads, exports every entry point that
include/salt.h declares, and its host-only functions agree with the oracle.
No GPU call is made here."""
import os
import re

import numpy as np

import oracle
from paper_2608_03579_amd import salt, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "salt.h")).read()
    return sorted(set(re.findall(r"SALT_API\s+[\w\s\*]+?\b(salt_\w+)\s*\(", src)))


def test_header_and_binding_agree():
    assert declared_symbols() == sorted(salt.EXPORTS)


def test_library_exports_every_declared_symbol():
    for name in declared_symbols():
        assert hasattr(salt.lib, name), name
    assert salt.lib.salt_version() == 1


def test_status_strings():
    for s in range(8):
        assert salt.lib.salt_status_str(s)
    assert salt.lib.salt_status_str(99) == b"unknown status"


def test_residual_bytes_matches_oracle_footprint():
    for cfg in (1, 2, 3, 4, 5):
        w = synth.make(cfg, 0)
        shapes = [(i, o) for _, i, o in w.tables]
        for r in (0, 1, 2, 16):
            want = oracle.adapter_bytes(r, shapes, 1, w.esize)
            got = salt.residual_bytes_for(salt.F32 if w.dtype == "f32" else salt.BF16, shapes, r)
            assert got == want, (cfg, r, got, want)
            assert got == r * w.blob_elems(1) * w.esize
    assert salt.residual_bytes_for(salt.BF16, [(3072, 3072)], -1) == 0


def test_create_rejects_bad_configs_before_touching_the_gpu():
    # validation happens before any HIP call, so these run without a device
    bad = [
        dict(tables=[(3072, 3071)]),                # out_dim not a multiple of 8
        dict(n_centroids=65),                       # C > 64
        dict(n_centroids=0, r_c=8),                 # rank without centroids
        dict(r_u_max=73),                           # above the largest residual rank (72)
        dict(max_tokens=0),
        dict(max_tokens=65537),                     # above the largest plan
        dict(n_slots=0),
    ]

    base = dict(dtype="bf16", tables=[(3072, 3072)], n_centroids=4, r_c=32, n_slots=8, r_u_max=2,
                max_tokens=64)
    for b in bad:
        kw = {**base, **b}
        try:
            salt.Context(**kw)
        except salt.SaltError as e:
            assert e.status in (salt.ERR_INVALID_ARG, salt.ERR_OUT_OF_RANGE), e
        else:
            raise AssertionError(f"accepted {b}")


def test_create_rejects_unknown_flags():
    cfg = salt.Config(salt.BF16, 1, (salt.Shape * 1)(salt.Shape(3072, 3072)), 4, 32, 8, 2, 64, 0, 2)
    h = salt.C.c_void_p()
    assert salt.lib.salt_create(salt.C.byref(cfg), salt.C.byref(h)) == salt.ERR_INVALID_ARG
    assert not h.value
