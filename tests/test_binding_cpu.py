"""The Python binding's own checks, on the CPU: the C ABI sees only pointers,
so the binding rejects tensors whose dtype, shape or device would let a
kernel read or write past a buffer, before anything reaches the library
(every call below raises during validation; no GPU is touched)."""
import pytest
import torch

from paper_2406_05955_amd import binding as ts

B, H, I, E = 2, 64, 96, 4


def ffn_args(**kw):
    a = dict(x=torch.zeros(B, H), w_gate=torch.zeros(I, H, dtype=torch.bfloat16),
             w_up=torch.zeros(I, H, dtype=torch.bfloat16), w_down_t=torch.zeros(I, H, dtype=torch.bfloat16))
    a.update(kw)
    return a


def moe_args(**kw):
    a = dict(x=torch.zeros(B, H), w_router=torch.zeros(E, H, dtype=torch.bfloat16),
             w_gate=torch.zeros(E, I, H, dtype=torch.bfloat16), w_up=torch.zeros(E, I, H, dtype=torch.bfloat16),
             w_down_t=torch.zeros(E, I, H, dtype=torch.bfloat16))
    a.update(kw)
    return a


FFN_CALLS = [
    lambda **a: ts.ffn_sparse(**a),
    lambda **a: ts.ffn_dense(**a),
    lambda **a: ts.ffn_sparse_act(act=ts.TS_ACT_RELU_GATE, tau=0.1, **a),
    lambda **a: ts.ffn_sparse_topk(keep=8, **a),
    lambda **a: ts.ffn_sparse_given(idx=torch.zeros(B, 4, dtype=torch.int32),
                                    count=torch.zeros(B, dtype=torch.int32), **a),
]


@pytest.mark.parametrize("call", FFN_CALLS)
def test_ffn_entry_points_reject_mismatched_tensors(call):
    bf = torch.bfloat16
    with pytest.raises(TypeError, match="x must be a float32"):
        call(**ffn_args(x=torch.zeros(B, H, dtype=bf)))
    with pytest.raises(TypeError, match="x must be a float32"):
        call(**ffn_args(x=torch.zeros(H)))
    with pytest.raises(TypeError, match="float32 or bfloat16"):
        call(**ffn_args(w_gate=torch.zeros(I, H, dtype=torch.float16)))
    with pytest.raises(ValueError, match="w_gate must be"):
        call(**ffn_args(w_gate=torch.zeros(I, H + 8, dtype=bf)))
    with pytest.raises(ValueError, match="w_up must match"):
        call(**ffn_args(w_up=torch.zeros(I - 1, H, dtype=bf)))
    with pytest.raises(ValueError, match="w_down_t must match"):
        call(**ffn_args(w_down_t=torch.zeros(I, H)))
    with pytest.raises(ValueError, match="out must be"):
        call(**ffn_args(), out=torch.zeros(B, H + 1))
    with pytest.raises(ValueError, match="out must be"):
        call(**ffn_args(), out=torch.zeros(B, H, dtype=bf))
    # well-formed host tensors: refused for not being device memory
    with pytest.raises(ValueError, match="contiguous device tensors"):
        call(**ffn_args())


def test_moe_rejects_mismatched_tensors():
    bf = torch.bfloat16
    with pytest.raises(ValueError, match="w_gate must be"):
        ts.moe_sparse(top_k=2, **moe_args(w_gate=torch.zeros(I, H, dtype=bf), w_up=torch.zeros(I, H, dtype=bf),
                                          w_down_t=torch.zeros(I, H, dtype=bf)))
    with pytest.raises(ValueError, match="w_router must be"):
        ts.moe_sparse(top_k=2, **moe_args(w_router=torch.zeros(E + 1, H, dtype=bf)))
    with pytest.raises(ValueError, match="w_router must be"):
        ts.moe_sparse(top_k=2, **moe_args(w_router=torch.zeros(E, H)))
    with pytest.raises(ValueError, match="w_down_t must match"):
        ts.moe_dense(top_k=2, **moe_args(w_down_t=torch.zeros(E, I, H - 8, dtype=bf)))
    with pytest.raises(ValueError, match="contiguous device tensors"):
        ts.moe_sparse(top_k=2, **moe_args())


def test_probe_buffer_checks():
    with pytest.raises(ValueError, match="smaller than src"):
        ts.probe_copy(torch.zeros(64), torch.zeros(63))
    with pytest.raises(ValueError, match="at least 4096"):
        ts.probe_read(torch.zeros(64), torch.zeros(100))
    with pytest.raises(ValueError, match="contiguous device tensors"):
        ts.probe_read(torch.zeros(64), torch.zeros(4096))
