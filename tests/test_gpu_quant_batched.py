"""GPU parity of the grouped activation quantization
(sherry_quantize_act_batched) against the CPU oracle's quantizer: int8 codes
and fp32 scales bit-exact, for several matrices of different row lengths in
one launch (register-held rows and two-pass rows, zero rows, outliers)."""
import sys

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _sh():
    import paper_2601_07892_amd as sh
    return sh


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


@pytest.mark.parametrize("shapes", [
    [(96, 2048), (16, 8192)],                       # the LLaMA-3.2-1B decode step
    [(3, 4), (1, 2052), (5, 3072), (2, 16388), (70, 132)],  # ragged, one two-pass matrix
])
def test_quantize_batched_bit_exact(dev, shapes):
    sh = _sh()
    print("[case] quantize batched", shapes, file=sys.stderr, flush=True)
    descs = (sh.sherry_quant_desc * len(shapes))()
    keep = []
    for i, (m, k) in enumerate(shapes):
        x = synth.activations(m, k, 81, "qb", i, outlier_frac=0.01)
        x[0, :] = 0.0  # an all-zero row: scale 0, codes 0
        xd = torch.from_numpy(x).to(dev)
        q = torch.full((m, k), 99, dtype=torch.int8, device=dev)
        sx = torch.full((m,), -1.0, dtype=torch.float32, device=dev)
        d = descs[i]
        d.x, d.q, d.x_scale, d.m, d.k = xd.data_ptr(), q.data_ptr(), sx.data_ptr(), m, k
        keep.append((x, xd, q, sx))
    rows, max_k = sh.sherry_quantize_act_batched_prepare(descs)
    assert rows == sum(m for m, _ in shapes) and max_k == max(k for _, k in shapes)
    assert [d.row_begin for d in descs] == list(np.cumsum([0] + [m for m, _ in shapes])[:-1])
    dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
    sh.sherry_quantize_act_batched(dd, len(shapes), rows, max_k)
    torch.cuda.synchronize()
    for x, xd, q, sx in keep:
        q_ref, sx_ref = oracle.quantize_act(x)
        assert np.array_equal(q.cpu().numpy(), q_ref)
        assert np.array_equal(sx.cpu().numpy().view(np.uint32), sx_ref.view(np.uint32))
