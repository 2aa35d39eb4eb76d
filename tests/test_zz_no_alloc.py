"""hcms_attention_backward_noalloc on the GPU, through the C ABI: the entry
point that keeps D = <dO, O> in the library's static scratch array instead of
a caller's workspace gives the gradients of hcms_attention_backward, bit for
bit, on two calls in a row (the second on a smaller input, so stale scratch
contents from the first call would show).  The size limit is checked on the
CPU (tests/test_abi.py).
"""
import pytest
import torch

from tests.gpu_util import bits, log

pytestmark = pytest.mark.gpu


def _data(S, H, d, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    q, k, v, do = (torch.randn(H, S, d, generator=g) for _ in range(4))
    return [x.to(dtype).cuda() for x in (q, k, v, do)]


@pytest.mark.parametrize("d,dtype", [(128, torch.bfloat16), (64, torch.float32)])
def test_noalloc_backward_equals_workspace_backward(hcms, d, dtype):
    scale = d ** -0.5
    # First call large, second smaller (fewer heads, ragged S): each must
    # match the workspace entry point on its own inputs.
    for S, H, chunks, seed in ((3000, 4, (3, 1), 1), (777, 2, (1, 1), 2)):
        log(f"[noalloc] S={S} H={H} d={d} {dtype} chunks={chunks}")
        q, k, v, do = _data(S, H, d, dtype, seed * 100 + d)
        out, lse = hcms.attention_lse(q, k, v, scale, chunks)
        ref = [t.clone() for t in hcms.attention_backward(q, k, v, out, do, lse, scale, chunks)]
        got = [torch.full_like(q, float("nan")) for _ in range(3)]
        hcms.attention_backward_noalloc(q, k, v, out, do, lse, scale, chunks, *got)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), got, ref):
            assert torch.equal(bits(a), bits(b)), (S, H, name)

