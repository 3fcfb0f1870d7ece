"""Two independent bf16 products in one launch of the 256 x 256 kernels (the
form the weight gradients share in an HVP: q/k/v with wo, and gate/up with the
down projection's token slices as a batched second product): each output must
carry the same bits as a launch of its own on the same kernel, and match the
fp64 product, for every operand layout, ragged shapes (edge tiles in M and N,
different K), one or two operand pairs and batched products."""
import numpy as np
import pytest

import synth
from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("tile", [6, 8])
@pytest.mark.parametrize("ak,bk", [(1, 1), (1, 0), (0, 1), (0, 0)])
@pytest.mark.parametrize("batches", [(1, 1), (1, 3)])
def test_gemm_pair_matches_single_launches(tile, ak, bk, batches):
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    say(f"gemm pair tile={tile} ak={ak} bk={bk} batches={batches}")
    rng = np.random.default_rng(11 + tile + 2 * ak + bk + 5 * batches[1])
    shapes = [(600, 520, 96, 2), (296, 264, 160, 1 if batches[1] == 1 else 2)]   # (M, N, K, operand pairs)

    def mk(z, r, c):
        return synth.bf16_round(rng.standard_normal((z, r, c)).astype(np.float32))

    def up(x, kmaj):
        y = x if kmaj else np.ascontiguousarray(np.transpose(x, (0, 2, 1)))
        return torch.from_numpy(np.ascontiguousarray(y)).cuda().to(torch.bfloat16)

    ops, want = [], []
    for (M, N, K, npairs), z in zip(shapes, batches):
        A, B = mk(z, M, K), mk(z, N, K)
        A2, B2 = (mk(z, M, K), mk(z, N, K)) if npairs == 2 else (None, None)
        w = np.einsum("zmk,znk->zmn", A.astype(np.float64), B.astype(np.float64))
        if npairs == 2:
            w += np.einsum("zmk,znk->zmn", A2.astype(np.float64), B2.astype(np.float64))
        want.append(0.5 * w)
        ops.append((up(A, ak), up(B, bk), None if A2 is None else up(A2, ak), None if B2 is None else up(B2, bk)))
    pair = [torch.full((z, M, N), float("nan"), device="cuda") for (M, N, _, _), z in zip(shapes, batches)]
    fd.testing_gemm_pair(*shapes[0][:3], *shapes[1][:3], ak, bk, (*ops[0], pair[0]), (*ops[1], pair[1]), 0.5, tile,
                         batches[0], batches[1])
    single = [torch.full((z, M, N), float("nan"), device="cuda") for (M, N, _, _), z in zip(shapes, batches)]
    for (M, N, K, _), z, (A, B, A2, B2), C in zip(shapes, batches, ops, single):
        fd.testing_gemm("bf16", M, N, K, z, ak, bk, A, B, A2, B2, C, 0, 0.5, tile)
    for q in range(2):
        p, s = pair[q].cpu().numpy(), single[q].cpu().numpy()
        assert np.array_equal(p, s), f"product {q}: {np.count_nonzero(p != s)} elements differ"
        err = np.abs(p.astype(np.float64) - want[q]).max() / np.abs(want[q]).max()
        assert err < 2e-6, (q, err)


def test_gemm_pair_rejects_other_tiles():
    torch = need_gpu()
    from paper_2602_00816_amd import fdhvp as fd
    z = torch.zeros(64 * 64, device="cuda", dtype=torch.bfloat16)
    c = torch.zeros(64 * 64, device="cuda")
    with pytest.raises(fd.FdhError):
        fd.testing_gemm_pair(64, 64, 64, 64, 64, 64, 1, 1, (z, z, None, None, c), (z, z, None, None, c), 1.0, 4)
