"""GPU parity of qmlp_linear_batch (the linears outside the MLP: attention
projections and LM head, Sec. 3.3 at 4 bits, 2 bits for the uniform-W2
comparison point of Sec. 5.2) against the oracle's y = W_hat x on binary16
inputs, at the bar max|y - y_ref| / max|y_ref| <= 1e-2; packing bit-exact."""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import bits_of

pytestmark = pytest.mark.gpu

Y_TOL = 1e-2


@pytest.fixture(scope="module")
def q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04238_amd as qm
    qm.library()
    return qm


@pytest.mark.parametrize("bits,n,k,L,M,g", [
    (4, 6144, 2560, 3, 1, 128),      # the Qwen3-4B q/k/v projection, three layers
    (4, 2560, 4096, 2, 1, 128),      # its o projection
    (2, 6144, 2560, 2, 1, 128),      # the same at 2 bits (uniform W2)
    (4, 704, 640, 5, 7, 64),         # ragged unit counts, several tokens
    (2, 640, 1600, 40, 2, 64),       # a full batch of 40
])
def test_linear_batch_matches_oracle(q, bits, n, k, L, M, g):
    print("\n[case] linear_batch bits %d n %d k %d L %d M %d g %d" % (bits, n, k, L, M, g), flush=True)
    Ws = [wl.linear_weight(n, k, i, wl.TID_QKV) for i in range(L)]
    xs = [wl.linear_input(M, k, i, wl.TID_QKV) for i in range(L)]
    pack = q.pack_w4 if bits == 4 else q.pack_w2
    ws = [pack(torch.from_numpy(W).cuda(), g) for W in Ws]
    x = torch.stack([torch.from_numpy(a.view(np.int16)).view(torch.float16) for a in xs]).cuda()
    y = q.linear_batch(ws, x)
    torch.cuda.synchronize()
    Y = bits_of(y)
    for i in sorted({0, L - 1}):
        qt = orc.quantize(Ws[i], bits, g)
        assert np.array_equal(ws[i].codes.cpu().numpy().view(np.uint32).reshape(n, -1), qt.packed())
        ref = orc.down_act(qt, xs[i])
        err = orc.max_rel_err(orc.act_to_f64(Y[i], False), ref)
        print("block %d max-rel %.2e" % (i, err))
        assert err <= Y_TOL


def test_linear_batch_lm_head_rows_sampled(q):
    """The Qwen3-4B LM head shape (151936 x 2560, one launch) at 4 bits; rows
    sampled against the oracle."""
    dims = wl.DECODERS["qwen3_4b"]
    n, k = dims.vocab, 2560
    print("\n[case] linear_batch LM head", n, k, flush=True)
    W = wl.linear_weight(n, k, 0, wl.TID_LM_HEAD)
    xb = wl.linear_input(1, k, 0, wl.TID_LM_HEAD)
    w = q.pack_w4(torch.from_numpy(W).cuda(), 128)
    x = torch.from_numpy(xb.view(np.int16)).view(torch.float16).cuda().reshape(1, 1, k)
    y = q.linear_batch([w], x)
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(n, size=512, replace=False)
    rows.sort()
    qt = orc.quantize(W[rows], 4, 128)
    ref = orc.down_act(qt, xb)
    got = orc.act_to_f64(bits_of(y)[0, 0, rows].reshape(1, -1), False)
    assert orc.max_rel_err(got, ref) <= Y_TOL
