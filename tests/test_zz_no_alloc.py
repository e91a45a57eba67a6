"""GPU: protokv_attend_static, the readout for callers that cannot allocate.

Its kernels keep the split partials (and the rotated query) in the library's
fixed device array instead of the workspace.  Through the C-ABI it must give
protokv_attend's result -- bitwise here, since the split count is the same --
on two calls in a row, the second with a smaller query, for bf16 KV with one
and with two query-row blocks, with rotary positions, and for float32 KV;
a shape whose partials cannot fit the array is refused before any launch.
Each test prints its case before any GPU step.
"""
import numpy as np
import pytest

from paper_2606_26762_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26762_amd import protokv as pk
    pk.lib()
    yield


def H():
    from tests import gpu_harness
    return gpu_harness


CASES = {
    "bf16, one row block": (dict(num_layers=2, num_kv_heads=2, num_q_heads=8, grid_h=7, grid_w=7, frames=12,
                                 window_frames=3, capacity=40, query_tokens=16), {}, (16, 5)),
    "bf16, two row blocks": (dict(num_layers=1, num_kv_heads=2, num_q_heads=16, grid_h=7, grid_w=7, frames=12,
                                  window_frames=3, capacity=40, query_tokens=40), {}, (40, 3)),
    "bf16, rotary positions": (dict(num_layers=2, num_kv_heads=2, num_q_heads=4, grid_h=6, grid_w=6, frames=10,
                                    window_frames=2, capacity=48, query_tokens=8), dict(rope_theta=1e4), (8, 2)),
}


@pytest.mark.parametrize("case", list(CASES))
def test_static_scratch_readout_equals_the_workspace_readout(case):
    import torch
    h = H()
    shape, pkw, tqs = CASES[case]
    wl = W.WORKLOADS["7b"].with_(**shape)
    h.log(f"case: attend_static {case}")
    pair = h.Pair(wl, **pkw)
    for _ in range(wl.frames):
        pair.step()
    pair.gpu.synthesize(0)
    rng = np.random.default_rng(12)
    for tq in tqs:
        q = torch.from_numpy(pair.query(rng, tq=tq)).to("cuda", pair.dtype).contiguous()
        o1, l1 = pair.gpu.attend(0, q)
        o2, l2 = pair.gpu.attend_static(0, q)
        torch.cuda.synchronize()
        d = float((o1.float() - o2.float()).abs().max())
        h.log(f"tq {tq}: max |attend - attend_static| {d:.2e}")
        assert d <= h.READOUT_ATOL and float((l1 - l2).abs().max()) <= h.LSE_ATOL
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
    # and against the oracle once more, through the static path
    pseudo = pair.oracle[0].synthesize()
    q = pair.query(rng, tq=tqs[-1])
    oo, ol = pair.oracle[0].attend(q, wl.num_kv_heads, pseudo)
    go, gl = pair.gpu.attend_static(0, torch.from_numpy(q).to("cuda", pair.dtype).contiguous())
    torch.cuda.synchronize()
    assert np.abs(go.float().cpu().numpy() - oo).max() <= h.READOUT_ATOL
    assert np.abs(gl.cpu().numpy() - ol).max() <= h.LSE_ATOL


def test_static_scratch_readout_float32():
    import torch
    h = H()
    wl = W.WORKLOADS["tiny"].with_(frames=12)
    h.log("case: attend_static float32 tiny")
    pair = h.Pair(wl)
    for _ in range(wl.frames):
        pair.step()
    pair.gpu.synthesize(0)
    rng = np.random.default_rng(13)
    for tq in (16, 7):
        q = torch.from_numpy(pair.query(rng, tq=tq)).to("cuda", torch.float32).contiguous()
        o1, l1 = pair.gpu.attend(0, q)
        o2, l2 = pair.gpu.attend_static(0, q)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_partials_beyond_the_array_are_refused():
    """512 kv heads x 512 query rows: one split's partials are 136 MB, above the
    64 MiB array; refused (E_UNSUPPORTED) before anything is launched."""
    import torch
    from paper_2606_26762_amd import protokv as pk
    h = H()
    h.log("case: attend_static refusal, 512 units x 512 rows")
    cfg = pk.default_config(num_layers=64, num_kv_heads=8, num_q_heads=64, grid_h=2, grid_w=2, window_frames=1,
                            capacity=4, max_query_tokens=64)
    cb = np.zeros((64 * 8, 2, 8, 16, 16), dtype=np.float32)
    g = pk.ProtoKV(cfg, cb)
    q = torch.zeros((64, 64, 64, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(pk.ProtoKVError) as e:
        g.attend_static(0, q)
    assert e.value.status == 2
    torch.cuda.synchronize()
