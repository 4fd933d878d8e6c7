"""The allocation-free weight gradient psw_conv_bwd_weight_noalloc against
the workspace entry point psw_conv_bwd_weight, through the C ABI: the same
kernels in the same order, so the results must be identical bit for bit.
Two calls in a row, the second on a smaller input (the shared scratch keeps
the first call's contents, which the second must not read), in fp32 and in
bf16 mode; and a shape whose scratch need exceeds the array is refused."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    from paper_1912_12675_amd import psw
    psw.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return psw


CASES = [
    # N, C, H, W, K, R, stride, pad, bias -- in call order: large, then smaller
    (128, 16, 32, 32, 16, 3, 1, 1, False),  # ResNet-20 group 1 at the benchmark's batch (256 split partial sums)
    (8, 32, 16, 16, 64, 3, 2, 1, True),     # a smaller stride-2 layer with bias
]


@pytest.mark.parametrize("bf16", [False, True], ids=["fp32", "bf16"])
def test_noalloc_matches_workspace_entry_point(P, oracle, bf16):
    rng = np.random.default_rng(4242)
    for N, C, H, W, K, R, st, pad, bias in CASES:
        print(f"noalloc wgrad {(N, C, H, W, K, R, st, pad)} bias={bias} bf16={bf16}", flush=True)
        P_ = (H + 2 * pad - R) // st + 1
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        dy = rng.standard_normal((N, K, P_, P_)).astype(np.float32)
        xg, dyg = torch.from_numpy(x).cuda(), torch.from_numpy(dy).cuda()
        dw_ref = torch.full((K, C, R, R), 7.0, device="cuda")
        dw = torch.full((K, C, R, R), -3.0, device="cuda")
        db_ref = torch.full((K,), 7.0, device="cuda") if bias else None
        db = torch.full((K,), -3.0, device="cuda") if bias else None
        P.psw_conv_bwd_weight(xg, dyg, dw_ref, st, pad, dbias=db_ref, bf16=bf16)
        P.psw_conv_bwd_weight_noalloc(xg, dyg, dw, st, pad, dbias=db, bf16=bf16)
        torch.cuda.synchronize()
        assert torch.equal(dw, dw_ref)
        if bias:
            assert torch.equal(db, db_ref)
        ref = oracle.conv_bwd_weight(x, (K, C, R, R), dy, st, pad, bias=bias, bf16=bf16)
        rdw = ref[0] if bias else ref
        err = np.abs(dw.double().cpu().numpy() - rdw).max() / np.abs(rdw).max()
        assert err <= 2e-5, err


def test_noalloc_refuses_oversize_shape(P):
    """A 3x3 conv 1024 -> 1024 needs 36 MiB of split partial sums: refused
    with PSW_ERR_WORKSPACE before anything is enqueued (dw keeps its value)."""
    N, C, H, W, K = 2, 1024, 4, 4, 1024
    assert P.lib().psw_conv_bwd_weight_ws_bytes(N, C, H, W, K, 3, 3, 1, 1, 0) > (32 << 20)
    x = torch.zeros((N, C, H, W), device="cuda")
    dy = torch.zeros((N, K, H, W), device="cuda")
    dw = torch.full((K, C, 3, 3), 5.0, device="cuda")
    with pytest.raises(P.PswError) as e:
        P.psw_conv_bwd_weight_noalloc(x, dy, dw, 1, 1)
    assert e.value.code == -6
    torch.cuda.synchronize()
    assert bool((dw == 5.0).all())
