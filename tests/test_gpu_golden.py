"""The hand-derived worked examples of tests/golden through the C ABI.

Each fixture is one sync step (Equation 3, Algorithm 2, the sync lines of
Algorithm 1) with its expected own and server packed words, scales, errors,
average and reconstructed momentum and model; the library must reproduce
every value bit for bit, with eager and deferred sync writes and with
binary32 and bfloat16 gradients (the examples' gradients are small integers,
exact in bfloat16).
"""
import numpy as np
import pytest

import golden_io

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _eq(got, want, what):
    got = got.detach().cpu().numpy() if hasattr(got, "detach") else np.asarray(got)
    if want.dtype == np.uint64:
        got = got.view(np.uint64)
    assert np.array_equal(got, want), f"{what}: {got} != {want}"


@pytest.mark.parametrize("grad_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("defer", [False, True])
@pytest.mark.parametrize("name", golden_io.names())
def test_worked_example(torch_cuda, name, defer, grad_dtype):
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    su, ex = golden_io.load(name)
    print(f"golden {name} defer={defer} grad={grad_dtype}", flush=True)
    n, W = su["segments"][-1], su["world"]
    f32 = dict(dtype=torch.float32, device="cuda")
    st = {k: torch.zeros(n, **f32) for k in ("x", "m", "v", "u", "err", "srv_err", "anchor")}
    st["x"].copy_(torch.from_numpy(su["x0"]))
    st["anchor"].copy_(st["x"])
    gt = {"f32": torch.float32, "bf16": torch.bfloat16}[grad_dtype]
    g = torch.from_numpy(su["g"]).to(device="cuda", dtype=gt)
    opt = zo.ZoAdam(beta1=su["beta1"], beta2=0.999, eps=su["eps"], world=W, chunk=su["chunk"],
                    seg_off=su["segments"], tv=[], tu=[0], state=st, defer_sync_writes=defer,
                    grad_dtype=grad_dtype)
    try:
        # init zeroes m, v, u and the errors (Algorithm 1's initial state);
        # the example then sets v, as an earlier interval would have
        st["v"].copy_(torch.from_numpy(su["v0"]))
        assert opt.num_chunks == 1
        nw = opt.packed_words
        packed = torch.zeros((W, nw), dtype=torch.int64, device="cuda")
        scales = torch.zeros((W, 1), **f32)
        opt.compress_pack_ef(0, su["gamma"], g, packed[0], scales[0])
        torch.cuda.synchronize()
        _eq(packed[0], ex["own_words"], "own words")
        _eq(scales[0], ex["own_scales"], "own scale")
        _eq(st["err"], ex["err"], "worker error")
        peers = torch.from_numpy(su["peer_words"].view(np.int64).reshape(W - 1, nw))
        packed[1:].copy_(peers)
        scales[1:, 0].copy_(torch.from_numpy(su["peer_scales"]))
        sp = torch.zeros(nw, dtype=torch.int64, device="cuda")
        ss = torch.zeros(1, **f32)
        avg = torch.zeros(n, **f32)
        opt.unpack_average(0, packed, scales, sp, ss, avg_debug=avg)
        torch.cuda.synchronize()
        _eq(avg, ex["avg"], "average")
        _eq(sp, ex["srv_words"], "server words")
        _eq(ss, ex["srv_scales"], "server scale")
        _eq(st["srv_err"], ex["srv_err"], "server error")
        assert opt.inexact_chunks() == 0
        opt.sync_update(0, sp, ss, None)
        torch.cuda.synchronize()
        _eq(opt.current("m"), ex["m"], "momentum")
        _eq(opt.current("x"), ex["x"], "model")
        _eq(opt.current("u"), np.zeros(n, np.float32), "buffer")
        _eq(st["v"], su["v0"], "variance")
        assert opt.gamma_sum == 0.0
    finally:
        opt.close()
