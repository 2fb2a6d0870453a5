"""flowmoe_gate_topk_bwd_noalloc, the gate backward for callers that cannot
allocate device memory, against flowmoe_gate_topk_bwd with a caller
workspace (the same kernels: bit-identical results) and against the oracle's
gate backward (Sec. 2.1's softmax gate Jacobian, dW_g = x^T dl, db, and the
dx term dl W_g^T). Two calls in a row share the library's static scratch,
the second with a smaller input, on both dW_g paths and both gate kinds."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_close, dev, host, need_gpu
from paper_2510_00207_amd import _lib as L

pytestmark = pytest.mark.gpu


def _case(T, M, E, k, gate, seed):
    rng = np.random.default_rng(seed)
    d = dev()
    bf = torch.bfloat16
    t = lambda a, dt=bf: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    x = t(rng.standard_normal((T, M)))
    wg = t(rng.standard_normal((M, E)) * 0.05)
    gl = (host(x) @ host(wg)).astype(np.float32).astype(np.float64)
    idx, w = oracle.topk_select(gl, k, gate)
    dtw = rng.standard_normal((T, k)).astype(np.float32)
    dx0 = t(rng.standard_normal((T, M)))
    s = L.make_shape(T, M, 8, E, k, 0, L.BF16, L.GELU, L.PACKED,
                     L.GATE_FULL if gate == "full" else L.GATE_RENORM)
    args = dict(x=x, wg=wg, gl=t(gl, torch.float32), idx=t(idx, torch.int32),
                w=t(w, torch.float32), dtw=t(dtw, torch.float32))
    return s, args, dx0, (idx, w.astype(np.float32).astype(np.float64), dtw.astype(np.float64), gl)


def _outputs(T, M, E, dx0):
    d = dev()
    return dict(dl=torch.full((T, E), 7.0, device=d), dwg=torch.full((M, E), 3.0, device=d),
                db=torch.full((E,), 3.0, device=d), dx=dx0.clone())


@pytest.mark.parametrize("gate", ["renorm", "full"])
@pytest.mark.parametrize("big,small", [
    ((3000, 1024, 64, 6), (1100, 520, 64, 4)),   # dW_g: MFMA kernel (renorm) / GEMM path (full)
    ((2000, 1024, 8, 2), (700, 264, 4, 2)),     # the same at E <= 16
])
def test_gate_bwd_noalloc_matches_workspace_call(gate, big, small):
    need_gpu()
    for n, (T, M, E, k) in enumerate((big, small)):
        s, a, dx0, (idx, w, dtw, gl) = _case(T, M, E, k, gate, seed=T + E + n)
        need = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
        assert 0 < need <= L.NOALLOC_SCRATCH_BYTES
        for acc in (0, 1):
            ref, got = _outputs(T, M, E, dx0), _outputs(T, M, E, dx0)
            ws = torch.empty(need, dtype=torch.uint8, device=dev())
            L.flowmoe_gate_topk_bwd(s, a["x"], a["wg"], a["gl"], a["idx"], a["w"], a["dtw"],
                                    ref["dl"], ref["dwg"], ref["db"], ref["dx"], acc, ws, need)
            L.flowmoe_gate_topk_bwd_noalloc(s, a["x"], a["wg"], a["gl"], a["idx"], a["w"],
                                            a["dtw"], got["dl"], got["dwg"], got["db"], got["dx"],
                                            acc)
            torch.cuda.synchronize()
            for key in ("dl", "dwg", "db", "dx"):
                assert torch.equal(got[key], ref[key]), (n, acc, key)
            g = oracle.gate_bwd(host(a["x"]), host(a["wg"]), idx, w, dtw, gl, gate)
            base = 3.0 if acc else 0.0
            assert_close(host(got["dl"]), g["d_logits"], "f32", "d_logits", tol=1e-5)
            assert_close(host(got["dwg"]) - base, g["dw_gate"], "bf16", "dw_gate")
            assert_close(host(got["db"]) - base, g["dbias"], "bf16", "dbias")
            assert_close(host(got["dx"]), host(dx0) + g["dx_gate"], "bf16", "dx + gate term")


def test_gate_bwd_noalloc_rejects_shapes_beyond_its_scratch():
    """A shape whose workspace exceeds the static scratch is an error raised
    before anything is enqueued (pointers are never dereferenced)."""
    s = L.make_shape(1 << 20, 1 << 17, 8, 64, 2, 0, L.BF16)
    assert L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD) > L.NOALLOC_SCRATCH_BYTES
    fake = 0x10000
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk_bwd_noalloc(s, fake, fake, None, fake, fake, fake, fake, fake, None,
                                        None, 0, stream=0)
    assert ei.value.status == L.ERR_WORKSPACE and "scratch" in str(ei.value)
