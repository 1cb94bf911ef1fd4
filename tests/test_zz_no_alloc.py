"""de_verify_layer_noalloc (the verify layer with its scratch in a static
device array) against de_verify_layer (the same layer with a caller
workspace), through the C ABI.

The two share every kernel, so every output must be identical: routing ids,
gates, the union and its lists bit for bit, and the layer output.  Two calls
in a row on the same GPU, the second with a smaller block, show that what the
first call left in the shared array does not leak into the second.  A shape
whose scratch exceeds the array is rejected before anything is enqueued.
"""
import numpy as np
import pytest
import torch

import paper_2607_24434_amd as de
from workloads import configs

from gpu_support import f32, layer_pair, require_gpu
from support import gapped_x

pytestmark = pytest.mark.gpu


def outputs(cfg, T):
    d = "cuda"
    return dict(
        y=torch.full((T, cfg.hidden), float("nan"), dtype=torch.float32, device=d),
        idx=torch.full((T, cfg.top_k), -7, dtype=torch.int32, device=d),
        gate=torch.full((T, cfg.top_k), float("nan"), dtype=torch.float32, device=d),
        nu=torch.full((1,), -7, dtype=torch.int32, device=d),
        uids=torch.full((cfg.n_experts,), -7, dtype=torch.int32, device=d),
        offs=torch.full((cfg.n_experts + 1,), -7, dtype=torch.int32, device=d),
        tok=torch.full((T * cfg.top_k,), -7, dtype=torch.int32, device=d),
        glist=torch.full((T * cfg.top_k,), float("nan"), dtype=torch.float32, device=d),
        ppos=torch.full((T, cfg.top_k), -7, dtype=torch.int32, device=d),
    )


def run(fn, dev, x, T, o, epi, **kw):
    fn(dev.desc, T, x, dev.router, dev.bias, dev.table, dev.shared, o["y"], o["idx"], o["gate"],
       o["nu"], o["uids"], o["offs"], o["tok"], o["glist"], o["ppos"], epi=epi, **kw)


@pytest.mark.parametrize("cfg,blocks", [(configs.CFG2, (17, 9)), (configs.CFG1, (5, 2))],
                         ids=["cfg2-T17-then-T9", "cfg1-T5-then-T2"])
def test_noalloc_verify_layer_equals_workspace_call(cfg, blocks):
    require_gpu()
    torch.cuda.set_device(0)
    orc, dev = layer_pair(cfg)
    for i, T in enumerate(blocks):
        x, _ = gapped_x(orc, T, block=10 + i)
        xd = f32(x)
        res = torch.randn(T, cfg.hidden, dtype=torch.float32, device="cuda")
        want, got = outputs(cfg, T), outputs(cfg, T)
        nw = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        ng = torch.empty(T, cfg.hidden, dtype=torch.float32, device="cuda")
        run(de.de_verify_layer, dev, xd, T, want, de.make_epilogue(residual=res, normed=nw),
            ws=dev.ws(T))
        run(de.de_verify_layer_noalloc, dev, xd, T, got, de.make_epilogue(residual=res, normed=ng))
        torch.cuda.synchronize()
        nu = int(want["nu"].item())
        print(f"{cfg.name} T={T}: union {nu}", flush=True)
        assert nu == len(set(orc.route(x)[0].ravel().tolist()))
        for k in ("idx", "gate", "nu", "tok", "glist", "ppos"):
            assert torch.equal(got[k], want[k]), k
        assert torch.equal(got["uids"][:nu], want["uids"][:nu])
        assert torch.equal(got["offs"][:nu + 1], want["offs"][:nu + 1])
        assert torch.equal(got["y"], want["y"])
        assert torch.equal(ng, nw)
        assert np.isfinite(got["y"].cpu().numpy()).all()


def test_noalloc_rejects_a_shape_beyond_its_scratch():
    require_gpu()
    big = de.make_desc(2048, 256, 32, 1408, 2816, 1408, 0, 0, 1.0, de.DE_BF16)
    assert de.de_workspace_bytes(big, 64) > de.de_noalloc_scratch_bytes()
    dummy = torch.empty(16, dtype=torch.float32, device="cuda")
    tab = de.make_table(dummy, 3 * 1408 * 2048 * 2, None, 256)
    with pytest.raises(de.DEError) as ei:
        de.de_verify_layer_noalloc(big, 64, dummy, dummy, None, tab, dummy, dummy)
    assert ei.value.code == -4
