"""ebrl_op_gemm_noalloc -- the GEMM entry point that allocates nothing --
against the allocating ebrl_op_gemm, through the C ABI: bitwise equal
outputs on shapes that split K (the decode kernel's in-kernel reduction, and
the K % 64 != 0 kernel with its reduce pass), on shapes that do not, and on
two calls in a row with the second smaller; a shape whose split would not fit
the fixed scratch array is refused.  Both also match the definition of the
product (the oracle's linear layer)."""
import numpy as np
import pytest

from oracle import model as M
from tests import parity as P

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2609_27547_amd import ebrl as E  # noqa: E402

SHAPES = [(200, 64, 16384), (130, 1024, 4096), (16, 256, 1032), (40, 8192, 1024), (17, 128, 72),
          (300, 1024, 512), (8, 4100, 11008)]


def _operands(m, n, k, dtype, seed):
    rng = np.random.default_rng(seed)
    a = torch.from_numpy(rng.normal(size=(m, k)).astype(np.float32))
    b = torch.from_numpy(rng.normal(size=(n, k)).astype(np.float32))
    if dtype == "bf16":
        a, b = a.to(torch.bfloat16), b.to(torch.bfloat16)
    return a.cuda(), b.cuda()


def _gemm(A, B, noalloc):
    C = torch.full((A.shape[0], B.shape[0]), float("nan"), dtype=torch.float32, device="cuda")
    E.op_gemm(A, B, C, noalloc=noalloc)
    return C


@pytest.mark.parametrize("m,n,k", SHAPES)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_noalloc_gemm_equals_allocating_entry_point(m, n, k, dtype):
    print(f"noalloc gemm {dtype} M={m} N={n} K={k}", flush=True)
    A, B = _operands(m, n, k, dtype, m + n + k)
    m2 = max(1, m // 3)
    A2 = A[:m2].contiguous()
    got = _gemm(A, B, True)
    got2 = _gemm(A2, B, True)          # second call in a row, smaller input
    ref = _gemm(A, B, False)
    ref2 = _gemm(A2, B, False)
    torch.cuda.synchronize()
    assert torch.equal(got, ref) and torch.equal(got2, ref2)
    a64 = A.float().cpu().numpy().astype(np.float64)
    b64 = B.float().cpu().numpy().astype(np.float64)
    assert P.row_rel_err(got.cpu().numpy(), M.linear(a64, b64)) < 2e-6


def test_noalloc_gemm_refuses_a_split_larger_than_its_scratch():
    # 200 x 4096 x 4104 splits K 13 ways over 200 x 4096 partial sums each
    # (10.6 M floats), more than the 16 MB array holds
    A, B = _operands(200, 4096, 4104, "bf16", 1)
    C = torch.zeros((200, 4096), dtype=torch.float32, device="cuda")
    rc = E.lib().ebrl_op_gemm_noalloc(E.DTYPE_BF16, A.data_ptr(), B.data_ptr(), C.data_ptr(), 200, 4096, 4104,
                                      torch.cuda.current_stream().cuda_stream)
    assert rc == -1
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(C)) == 0
    # the allocating entry point takes it
    E.op_gemm(A, B, C)
    torch.cuda.synchronize()
    a64 = A.float().cpu().numpy().astype(np.float64)
    b64 = B.float().cpu().numpy().astype(np.float64)
    assert P.row_rel_err(C.cpu().numpy(), M.linear(a64, b64)) < 2e-6
