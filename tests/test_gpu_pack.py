"""GPU parity of moe_quant_pack against the oracle: codes and {scale, zero}
words must be identical bit for bit (Sec. IV-A quantizer, Sec. V-B packing)."""
import numpy as np
import pytest
import torch

from gpu_util import dev

pytestmark = pytest.mark.gpu


def _weights(rng, R, K, kind):
    if kind == "normal":
        return (rng.standard_normal((R, K)) * 0.02).astype(np.float32)
    if kind == "edge":
        w = (rng.standard_normal((R, K)) * 0.02).astype(np.float32)
        w[0] = 0.0                                    # degenerate groups
        w[1] = np.abs(w[1])                           # all positive
        w[2] = -np.abs(w[2])                          # all negative
        w[3] *= 1e-7                                  # subnormal fp16 scales
        w[4, ::7] = 3.0                               # outliers
        w[5] = 0.37                                   # constant
        return w
    raise ValueError(kind)


def _gpu_pack(w, bits, group, rows=None):
    import paper_2503_21135_amd as P
    R, K = w.shape
    n = R if rows is None else len(rows)
    codes = torch.zeros(n * K * bits // 32, dtype=torch.int32, device=dev())
    sz = torch.zeros(n * (K // group), dtype=torch.int32, device=dev())
    st = torch.zeros(1, dtype=torch.int32, device=dev())
    rt = None if rows is None else torch.tensor(rows, dtype=torch.int32, device=dev())
    P.moe_quant_pack(torch.from_numpy(w).to(dev()), bits, group, codes, sz, n=n, rows=rt,
                     ld_codes=K * bits // 32, sz_row_stride=K // group, sz_group_stride=1,
                     status=st)
    torch.cuda.synchronize()
    return (codes.cpu().numpy().view(np.uint32).reshape(n, -1),
            sz.cpu().numpy().view(np.uint32).reshape(n, -1), int(st.item()))


@pytest.mark.parametrize("bits,group", [(2, 64), (4, 64), (8, 64), (2, 128), (3, 128),
                                        (4, 128), (6, 128), (8, 128)])
@pytest.mark.parametrize("kind", ["normal", "edge"])
def test_pack_bitexact(orc, bits, group, kind):
    rng = np.random.default_rng(bits * 100 + group)
    R, K = 40, 1408 if group == 128 else 512
    w = _weights(rng, R, K, kind)
    codes, sz, st = _gpu_pack(w, bits, group)
    assert st == 0
    s, q, s16, z16 = orc.quantize(w, bits, group)
    assert s == 0
    assert np.array_equal(codes, orc.pack(q, bits))
    assert np.array_equal(sz, orc.sz_words(s16, z16))


def test_pack_row_subset_and_overflow(orc):
    rng = np.random.default_rng(9)
    w = (rng.standard_normal((64, 256)) * 0.02).astype(np.float32)
    rows = [63, 0, 17, 17, 5]
    codes, sz, st = _gpu_pack(w, 8, 64, rows)
    s, q, s16, z16 = orc.quantize(w[rows], 8, 64)
    assert st == 0
    assert np.array_equal(codes, orc.pack(q, 8))
    assert np.array_equal(sz, orc.sz_words(s16, z16))
    w[3, 5] = 1e9
    _, _, st = _gpu_pack(w, 2, 64)
    assert st == -6


@pytest.mark.parametrize("name", ["mixtral-decode", "deepseek-decode"])
def test_pack_full_size_sampled_rows(orc, name):
    """Full-size expert matrices: GPU pack of whole matrices, sampled rows
    compared with the oracle."""
    import moe_inputs as mi
    inp = mi.LayerInputs(mi.WORKLOADS[name].layer)
    rng = np.random.default_rng(1)
    E = inp.cfg.n_experts
    for e in (0, E - 1):
        b = int(inp.bits[e])
        for kind in (0, 2):
            w = inp.weight(e, kind)
            codes, sz, st = _gpu_pack(w, b, inp.cfg.group)
            assert st == 0
            rows = np.sort(rng.choice(w.shape[0], 64, replace=False))
            s, q, s16, z16 = orc.quantize(w[rows], b, inp.cfg.group)
            assert np.array_equal(codes[rows], orc.pack(q, b))
            assert np.array_equal(sz[rows], orc.sz_words(s16, z16))
