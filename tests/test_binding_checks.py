"""The Python binding checks every tensor before it calls the library (CPU, no GPU needed).

A tensor on the wrong device, of the wrong dtype or shape, or not contiguous would make
the kernels read or write out of bounds; the binding raises instead, before any C call.
These tests use a plan object whose library handle is a tripwire: any C call fails the
test.  The device predicate is widened to accept CPU tensors where a test needs to reach
the dtype and shape checks behind it.
"""

import pytest
import torch

import paper_2606_01813_amd as pkg
from paper_2606_01813_amd import Plan, TreeOutputs

B, L, V, K, CAP = 3, 4, 64, 4, 40


class _Tripwire:
    def __getattr__(self, name):
        raise AssertionError(f"the library was called ({name}) before the arguments were checked")


def _plan(mask="u8", cap=CAP):
    p = object.__new__(Plan)
    p.L, p.V, p.K, p.cap, p.dtype, p.mask = L, V, K, cap, "f32", mask
    p.device = 0
    p._lib = _Tripwire()
    p._h = None
    return p


def _outputs(b=B, cap=CAP, mask="u8", topk=True):
    i32, f32 = dict(dtype=torch.int32), dict(dtype=torch.float32)
    m = None
    if mask == "u8":
        m = torch.zeros((b, cap, cap), dtype=torch.uint8)
    elif mask == "bits":
        m = torch.zeros((b, cap, (cap + 31) // 32), dtype=torch.int32)
    out = TreeOutputs(token_ids=torch.zeros((b, cap), **i32), parent=torch.zeros((b, cap), **i32),
                      depth=torch.zeros((b, cap), **i32), path_prob=torch.zeros((b, cap), **f32),
                      n_star=torch.zeros((b,), **i32), phi=torch.zeros((b,), **f32), theta=torch.zeros((b,), **f32),
                      mask=m, pos_ids=torch.zeros((b, cap), **i32))
    if topk:
        out.topk_ids = torch.zeros((b, L, K), **i32)
        out.topk_logit = torch.zeros((b, L, K), **f32)
        out.topk_lq = torch.zeros((b, L, K), **f32)
        out.lse = torch.zeros((b, L), dtype=torch.float64)
    return out


@pytest.fixture
def cpu_is_device(monkeypatch):
    monkeypatch.setattr(pkg, "_on_device", lambda t, device: t.device.type == "cpu")


def _logits(b=B):
    return torch.zeros((b, L, V), dtype=torch.float32)


def test_host_tensors_are_rejected():
    p = _plan()
    with pytest.raises(ValueError, match="cuda:0"):
        p.build(_logits(), _outputs())
    with pytest.raises(ValueError, match="cuda:0"):
        p.reduce_topk(_logits(), *[_outputs().__dict__[k] for k in ("topk_ids", "topk_logit", "lse")])
    o = _outputs()
    with pytest.raises(ValueError, match="cuda:0"):
        p.expand(o.topk_ids, o.topk_logit, o.lse, o)
    with pytest.raises(ValueError, match="cuda:0"):
        p.emit(o)


def test_non_tensors_are_rejected(cpu_is_device):
    p = _plan()
    with pytest.raises(TypeError):
        p.build(_logits().numpy(), _outputs())
    o = _outputs()
    o.parent = o.parent.numpy()
    with pytest.raises(TypeError):
        p.build(_logits(), o)


@pytest.mark.parametrize("field,bad", [
    ("token_ids", lambda o: o.token_ids[:2]),                             # fewer rounds than the logits
    ("parent", lambda o: torch.zeros((B, CAP - 1), dtype=torch.int32)),   # not the plan's cap
    ("depth", lambda o: o.depth.to(torch.int64)),                         # dtype
    ("n_star", lambda o: torch.zeros((B, 1), dtype=torch.int32)),         # rank
    ("path_prob", lambda o: o.path_prob.t().contiguous().t()),            # not contiguous
    ("phi", lambda o: o.phi.to(torch.float64)),
    ("theta", lambda o: o.theta[:1]),
    ("pos_ids", lambda o: torch.zeros((B, 2 * CAP), dtype=torch.int32)),
    ("mask", lambda o: torch.zeros((B, CAP, CAP - 1), dtype=torch.uint8)),
    ("mask", lambda o: torch.zeros((B, CAP, CAP), dtype=torch.int8)),
    ("topk_ids", lambda o: torch.zeros((B, L, K + 1), dtype=torch.int32)),
    ("topk_logit", lambda o: torch.zeros((B, L + 1, K), dtype=torch.float32)),
    ("topk_lq", lambda o: torch.zeros((B, L, K), dtype=torch.float64)),
    ("lse", lambda o: torch.zeros((B, L), dtype=torch.float32)),
    ("token_ids", lambda o: None),                                        # required
])
def test_build_rejects_bad_outputs(cpu_is_device, field, bad):
    p = _plan()
    o = _outputs()
    setattr(o, field, bad(o))
    with pytest.raises((ValueError, TypeError)):
        p.build(_logits(), o)


@pytest.mark.parametrize("mask,shape,dtype", [
    ("bits", (B, CAP, CAP), torch.int32),                 # a dense-shaped buffer for a packed mask
    ("bits", (B, CAP, 1), torch.int32),                   # too few words per row
    ("bits", (B, CAP, (CAP + 31) // 32), torch.uint8),
    ("u8", (B, CAP, (CAP + 31) // 32), torch.int32),      # a packed buffer for a dense mask
])
def test_mask_layout_must_match_the_plan(cpu_is_device, mask, shape, dtype):
    p = _plan(mask=mask)
    o = _outputs(mask=mask)
    o.mask = torch.zeros(shape, dtype=dtype)
    with pytest.raises((ValueError, TypeError)):
        p.build(_logits(), o)
    with pytest.raises((ValueError, TypeError)):
        p.emit(o)


def test_logits_checks(cpu_is_device):
    p = _plan()
    with pytest.raises(TypeError):
        p.build(torch.zeros((B, L, V), dtype=torch.bfloat16), _outputs())
    with pytest.raises(ValueError):
        p.build(torch.zeros((B, L + 1, V), dtype=torch.float32), _outputs())
    with pytest.raises(ValueError):
        p.build(torch.zeros((B, L, V - 1), dtype=torch.float32), _outputs())
    with pytest.raises(ValueError):
        p.build(torch.zeros((B, V, L), dtype=torch.float32).transpose(1, 2), _outputs())


def test_workspace_and_ctx_checks(cpu_is_device, monkeypatch):
    p = _plan()
    o = _outputs()
    monkeypatch.setattr(pkg, "_on_device", lambda t, device: t.device.type == "cpu" and t.numel() != 1024)
    with pytest.raises(ValueError, match="workspace"):
        p.build(_logits(), o, workspace=torch.zeros(1024, dtype=torch.uint8))
    monkeypatch.setattr(pkg, "_on_device", lambda t, device: t.device.type == "cpu")
    for bad in (torch.zeros(B, dtype=torch.int32), torch.zeros(B + 1, dtype=torch.int64),
                torch.zeros((B, 2), dtype=torch.int64)[:, 0]):
        with pytest.raises((ValueError, TypeError)):
            p.build(_logits(), o, ctx_len=bad)


def test_stage_calls_check_their_tables(cpu_is_device):
    p = _plan()
    o = _outputs()
    with pytest.raises(ValueError):
        p.reduce_topk(_logits(), o.topk_ids[:1], o.topk_logit, o.lse)
    with pytest.raises(ValueError):
        p.expand(o.topk_ids, o.topk_logit[:2], o.lse, o)
    small = _outputs(b=2)
    with pytest.raises(ValueError):
        p.expand(o.topk_ids, o.topk_logit, o.lse, small)          # outputs for fewer rounds
    o2 = _outputs()
    o2.n_star = o2.n_star[:1]
    with pytest.raises(ValueError):
        p.emit(o2)


def test_accept_checks(cpu_is_device):
    p = _plan()
    o = _outputs()
    u = torch.zeros((B, L), dtype=torch.float64)
    al = torch.zeros(B, dtype=torch.int32)
    with pytest.raises(ValueError):
        p.accept(o, o, u[:, :2].contiguous(), al)
    with pytest.raises(TypeError):
        p.accept(o, o, u.to(torch.float32), al)
    with pytest.raises(ValueError):
        p.accept(o, o, u, al[:1])
    o2 = _outputs()
    o2.parent = torch.zeros((B, CAP + 1), dtype=torch.int32)
    with pytest.raises(ValueError):
        p.accept(o, o2, u, al)
    o3 = _outputs()
    o3.token_ids = torch.zeros(B * CAP, dtype=torch.int32)
    with pytest.raises(ValueError):
        p.accept(o, o3, u, al)


def test_valid_arguments_reach_the_library(cpu_is_device):
    """With every argument valid the checks pass and the call goes on to the library (the tripwire)."""
    p = _plan()
    with pytest.raises(AssertionError, match="library was called"):
        p.build(_logits(), _outputs())
    bits = _plan(mask="bits")
    with pytest.raises(AssertionError, match="library was called"):
        bits.build(_logits(), _outputs(mask="bits"))
    o = _outputs()
    with pytest.raises(AssertionError, match="library was called"):
        p.expand(o.topk_ids, o.topk_logit, o.lse, o)
    with pytest.raises(AssertionError, match="library was called"):
        p.emit(o)
