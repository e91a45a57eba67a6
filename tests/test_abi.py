"""The C-ABI library loads, exports every symbol protokv.h declares, and its
host-only entry points (defaults, validation, workspace sizing) behave as
documented.  No GPU is touched."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_26762_amd import protokv as pk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "protokv.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:protokv_status|const char\*)\s+(protokv_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["protokv_init", "protokv_append_frame", "protokv_fold", "protokv_synthesize",
                     "protokv_attend"]:
        assert required in names
    assert sorted(pk.EXPORTED) == names


def test_library_exports_every_declared_symbol():
    lib = pk.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", pk.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (protokv_\w+)", out))
    assert set(declared_functions()) <= exported


def test_default_config_is_table5():
    c = pk.default_config()
    assert (c.pseudo_per_proto, c.pq_subspaces, c.pq_codewords, c.beam) == (8, 8, 16, 32)
    assert (c.lambda_sp, c.lambda_idle, c.t_idle) == (0.1, 0.01, 120)
    assert abs(c.eta - 0.05) < 1e-8 and c.pq_eps == 1.0
    assert abs(c.alpha - 0.05) < 1e-8 and abs(c.beta - 0.05) < 1e-8
    assert c.flags == pk.FLAG_PQ | pk.FLAG_MASS_BIAS
    assert lib_status(c) == 0


def lib_status(c):
    return pk.lib().protokv_validate_config(ctypes.byref(c))


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 64, 2), ("num_q_heads", 30, 1), ("num_streams", 0, 1), ("pq_subspaces", 4, 2),
    ("pq_codewords", 17, 2), ("pseudo_per_proto", 17, 2), ("beam", 4, 1), ("capacity", 0, 1),
    ("window_frames", 0, 1), ("grid_h", 80, 2), ("kv_dtype", 7, 1), ("flags", 64, 1),
    ("eta", 0.0, 1), ("pq_eps", 0.5, 2), ("ridge", 0.0, 1), ("lambda_sp", -1.0, 1),
    ("max_query_tokens", 100, 2), ("max_query_tokens", 0, 1), ("t_idle", -1, 1),
    ("rope_theta", 0.5, 1), ("rope_theta", -1.0, 1), ("rope_theta", float("inf"), 1),
    ("warm_frames", -1, 1),
])
def test_validation_rejects(field, value, status):
    c = pk.default_config(**{field: value})
    assert lib_status(c) == status
    assert pk.lib().protokv_last_error(None)


@pytest.mark.parametrize("kw,status", [
    (dict(alpha=1.5), 1), (dict(beta=-0.1), 1), (dict(flags=pk.FLAG_MAINTENANCE), 2), ({}, 0),
])
def test_ema_centre_validation(kw, status):
    """EMA rates must lie in [0, 1]; EMA centres with maintenance are not
    supported."""
    flags = pk.FLAG_PQ | pk.FLAG_MASS_BIAS | pk.FLAG_EMA_CENTRES | kw.pop("flags", 0)
    assert lib_status(pk.default_config(flags=flags, **kw)) == status


@pytest.mark.parametrize("kw,status", [
    (dict(warm_tokens=0), 1), (dict(kmeans_epochs=0), 1), (dict(kmeans_batch=65), 1),
    (dict(flags=pk.FLAG_MASS_BIAS), 1), (dict(flags=pk.FLAG_PQ | pk.FLAG_EMA_CENTRES), 2), ({}, 0),
])
def test_warmup_validation(kw, status):
    """Warm-up sizes must be positive (batch at most 64), it needs PQ and
    does not combine with EMA centres."""
    assert lib_status(pk.default_config(warm_frames=2, **kw)) == status


def test_workspace_size_scales_with_shape():
    small = pk.workspace_size(pk.default_config(num_layers=1, num_kv_heads=1, num_q_heads=1))
    full = pk.workspace_size(pk.default_config())
    multi = pk.workspace_size(pk.default_config(num_streams=4))
    assert 0 < small < full < multi
    # rings + banks dominate: 112 units x (9 frames x 196 x 128 x 2 x 2 B + 256 x 3200 B)
    assert full > 112 * (9 * 196 * 128 * 4 + 256 * 3200)
    with pytest.raises(pk.ProtoKVError):
        pk.workspace_size(pk.default_config(head_dim=96))


def test_state_header_and_bank_encoding_round_trip():
    """The state header is 128 bytes with the documented field order, and the
    bank encoder writes the documented row layout that decode_bank reads."""
    import ctypes
    import numpy as np
    assert ctypes.sizeof(pk.StateHeader) == 128
    assert pk.StateHeader.off_ring_k.offset == 72 and pk.StateHeader.total_bytes.offset == 120
    rng = np.random.default_rng(0)
    U, K = 3, 5
    bank = {"sum_k": rng.standard_normal((U, K, 128)).astype(np.float32),
            "sum_v": rng.standard_normal((U, K, 128)).astype(np.float32),
            "sq_k": rng.random((U, K, 128)).astype(np.float32),
            "sq_v": rng.random((U, K, 128)).astype(np.float32),
            "hist_k": rng.integers(0, 9, (U, K, 8, 12)).astype(np.uint32),
            "hist_v": rng.integers(0, 9, (U, K, 8, 12)).astype(np.uint32),
            "n": rng.integers(0, 99, (U, K)).astype(np.uint32),
            "n_res": rng.integers(0, 99, (U, K)).astype(np.uint32),
            "mu": rng.random((U, K, 2)).astype(np.float32),
            "sigma": rng.random((U, K, 3)).astype(np.float32),
            "tau": rng.integers(0, 999, (U, K)).astype(np.int32)}
    raw = pk.encode_bank(bank, U, K)
    assert raw.size == U * K * 3200
    back = pk.decode_bank(raw, U, K)
    for name, want in bank.items():
        got = back[name][..., :want.shape[-1]] if name.startswith("hist") else back[name]
        assert np.array_equal(got, want), name
    assert not back["hist_k"][..., 12:].any()
    # field offsets of the documented row
    row = raw.reshape(U, K, 3200)[1, 2]
    assert row[3072:3076].view(np.uint32)[0] == bank["n"][1, 2]
    assert row[3100:3104].view(np.int32)[0] == bank["tau"][1, 2]
    assert np.array_equal(row[512:1024].view(np.float32), bank["sum_v"][1, 2])


@pytest.mark.parametrize("kw,status", [
    (dict(pseudo_max=7), 1), (dict(pseudo_max=17), 2), (dict(capacity=5000), 2), (dict(beam=12), 1), ({}, 0),
    (dict(pseudo_max=8), 0), (dict(capacity=4096), 0)])
def test_variance_allocation_validation(kw, status):
    """The variance-aware allocation needs S <= pseudo_max <= 16, a beam of at
    least pseudo_max, and a capacity of at most 4096."""
    flags = pk.FLAG_PQ | pk.FLAG_MASS_BIAS | pk.FLAG_VAR_ALLOC
    assert lib_status(pk.default_config(flags=flags, **kw)) == status
    assert pk.default_config().pseudo_max == 16
