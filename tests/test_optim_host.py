"""Host-side rules of the torch.optim front end (CPU: no kernel runs)."""
import pytest
import torch

from paper_2607_10611_amd.optim import MAdam


def test_constructor_rejects_bad_options():
    p = [torch.nn.Parameter(torch.zeros(4, dtype=torch.bfloat16))]
    with pytest.raises(ValueError, match="rounding"):
        MAdam(p, rounding="nearest")
    with pytest.raises(ValueError, match="state_format"):
        MAdam(p, state_format="fp16")
    with pytest.raises(ValueError, match="betas"):
        MAdam(p, betas=(0.9,))


def test_global_index_bases_follow_parameter_order_across_groups():
    ps = [torch.nn.Parameter(torch.zeros(n, dtype=torch.bfloat16)) for n in (3, 5, 7, 11)]
    opt = MAdam([{"params": ps[:2]}, {"params": ps[2:3], "lr_add": 1e-2}])
    opt.add_param_group({"params": ps[3:]})
    assert [opt._base[p] for p in ps] == [0, 3, 8, 15]


def test_step_refuses_host_tensors_and_unsupported_dtypes_before_any_call():
    p = torch.nn.Parameter(torch.zeros(8, dtype=torch.bfloat16))
    p.grad = torch.zeros(8, dtype=torch.bfloat16)
    opt = MAdam([p])
    with pytest.raises(ValueError, match="GPU tensor"):
        opt.step()
    assert not opt.state[p]  # no state was made
    q = torch.nn.Parameter(torch.zeros(8, dtype=torch.float16))
    q.grad = torch.zeros(8, dtype=torch.float16)
    with pytest.raises(TypeError, match="no storage format"):
        MAdam([q]).step()
    r = torch.nn.Parameter(torch.zeros(8, dtype=torch.bfloat16))
    r.grad_dtype = None  # allow a gradient dtype other than the parameter's
    r.grad = torch.zeros(8, dtype=torch.float64)
    with pytest.raises(TypeError, match="gradients of dtype"):
        MAdam([r]).step()


def test_step_without_gradients_is_a_no_op():
    p = torch.nn.Parameter(torch.zeros(8, dtype=torch.bfloat16))
    opt = MAdam([p])
    assert opt.step() is None
    assert opt.step(lambda: 3.0) == 3.0
    assert not opt.state[p]


def test_master_format_rules():
    p = [torch.nn.Parameter(torch.zeros(128, dtype=torch.bfloat16))]
    with pytest.raises(ValueError, match="master_format"):
        MAdam(p, master_format="fp4")
    with pytest.raises(ValueError, match="master_format"):
        MAdam([{"params": p, "master_format": "e3m4"}])
    q = torch.nn.Parameter(torch.zeros(128))
    q.grad = torch.zeros(128)
    with pytest.raises(TypeError, match="compute copy"):
        MAdam([q], master_format="e4m3").step()       # the parameter holds the bf16 copy
    r = torch.nn.Parameter(torch.zeros(100, dtype=torch.bfloat16))
    r.grad = torch.zeros(100, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="multiple of 32"):
        MAdam([r], master_format="mxfp4").step()
    s = torch.nn.Parameter(torch.zeros(64, dtype=torch.bfloat16))
    s.grad = torch.zeros(64, dtype=torch.bfloat16)
    with pytest.raises(TypeError, match="float32"):
        MAdam([s], master_format="nvfp4_current").step()


def test_capturable_rules():
    p = [torch.nn.Parameter(torch.zeros(8, dtype=torch.bfloat16)) for _ in range(2)]
    with pytest.raises(RuntimeError, match="capturable"):
        MAdam(p).prepare_replay()
    p[1].grad = torch.zeros(8, dtype=torch.bfloat16)   # p[0] has none
    with pytest.raises(ValueError, match="needs a gradient"):
        MAdam(p, capturable=True).step()
    MAdam(p, capturable=True).prepare_replay()         # nothing stepped yet: nothing to do
