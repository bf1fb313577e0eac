"""moe_expert_ffn_mixed_noalloc -- the expert FFN on the library's fixed
per-GPU workspace, for callers that cannot allocate -- called through the C
ABI and compared with moe_expert_ffn_mixed on a caller workspace: the same
kernels on the same inputs, so the outputs must agree bit for bit.  Two calls
in a row, the second with a smaller batch (the fixed array still holds the
first call's contents), then a batch too large for the array."""
import ctypes as C

import numpy as np
import pytest
import torch

import moe_inputs as mi
from gpu_util import rel_l2, to_dev_bf16

pytestmark = pytest.mark.gpu


def _p(t):
    return C.c_void_p(t.data_ptr())


def test_noalloc_matches_workspace_entry(orc):
    import paper_2503_21135_amd as P
    from paper_2503_21135_amd import _lib
    lib = _lib.load()
    wk = mi.WORKLOADS["deepseek-decode"]
    cfg = wk.layer
    inp = mi.LayerInputs(cfg)
    layer = P.MoELayer(inp)
    layer.set_epoch(0)
    rs = orc.switch_state(inp, 0)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    for T in (128, 40):
        x_bits = mi.make_x(cfg, T, stream=1200 + T)
        x = to_dev_bf16(x_bits)
        b = layer.route(x)
        o_ref = torch.full_like(b.o, float("nan"))
        o_na = torch.full_like(b.o, float("nan"))
        ws = b.ffn_ws
        st = lib.moe_expert_ffn_mixed(C.byref(layer.desc), _p(x), T, cfg.top_k, _p(b.offsets),
                                      _p(b.perm), _p(o_ref), _p(ws), ws.numel(), None, stream)
        assert st == 0
        st = lib.moe_expert_ffn_mixed_noalloc(C.byref(layer.desc), _p(x), T, cfg.top_k,
                                              _p(b.offsets), _p(b.perm), _p(o_na), None, stream)
        assert st == 0
        torch.cuda.synchronize()
        assert torch.equal(o_ref, o_na), "T=%d: outputs differ" % T
        # the layer output from the no-allocation call against the oracle
        b.o.copy_(o_na)
        y = layer.combine(b).cpu().numpy()
        toks = np.arange(0, T, 5)
        res = orc.layer_forward(inp, x_bits, row_slot=rs, tokens=toks)
        err = rel_l2(y[toks], res["y"])
        print("no-alloc FFN T=%d: bitwise equal to the workspace call; rel L2 vs oracle %.3g"
              % (T, err), flush=True)
        assert err <= 5e-4
    # a batch whose workspace exceeds the fixed array is refused, nothing launched
    T = 16
    while True:
        _, need = P.api.moe_ffn_plan(layer.desc, T, cfg.top_k)
        if need > _lib.NOALLOC_SCRATCH_BYTES:
            break
        T *= 2
    dummy = torch.empty(16, dtype=torch.int32, device="cuda")
    st = lib.moe_expert_ffn_mixed_noalloc(C.byref(layer.desc), _p(dummy), T, cfg.top_k, _p(dummy),
                                          _p(dummy), _p(dummy), None, stream)
    assert st == _lib.ERR_WORKSPACE
