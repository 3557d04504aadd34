"""hp_stage_backward_noalloc (the backward pass on the library's static
scratch, for callers that cannot allocate) against hp_stage_backward on the
same stage and inputs: bit for bit, on two calls in a row, the second with a
smaller input (the scratch then holds the first call's partials)."""
import numpy as np
import pytest
import torch

from oracle import nets as onets
from paper_2005_14038_amd import hetpipe as hp

from gpu_common import dev  # noqa: F401
from stage_harness import make_inputs, oracle_weights, to_layers

pytestmark = pytest.mark.gpu


def _mid(H, groups):
    return onets.resnet152_mid(H, H, groups=groups)


CASES = [
    # (name, network, batch, dtype): the second is smaller than the first
    ("resnet-mid-16-fp32", lambda: _mid(16, [(128, 2, 2), (256, 2, 2)]), 2, "fp32"),
    ("resnet-mid-8-bf16", lambda: _mid(8, [(128, 1, 2), (256, 1, 2)]), 1, "bf16"),
    ("tiny-fp32", lambda: onets.tiny(8, 8), 1, "fp32"),
]


def _run(st, net, B, w, x, lab, dy, noalloc):
    grad = torch.full((st.P,), float("nan"), dtype=torch.float32, device="cuda")
    dx = torch.full(x.shape, float("nan"), dtype=torch.float32, device="cuda")
    if net.has_loss:
        y = torch.empty((B, net.nodes[-1]["classes"]), dtype=torch.float32, device="cuda")
        loss = torch.empty(1, dtype=torch.float32, device="cuda")
        st.forward(w, x, y, lab, loss)
        (st.backward_noalloc if noalloc else st.backward)(w, None, dx, grad)
    else:
        y = torch.empty((B,) + tuple(net.out_shape), dtype=torch.float32, device="cuda")
        st.forward(w, x, y)
        (st.backward_noalloc if noalloc else st.backward)(w, dy, dx, grad)
    torch.cuda.synchronize()
    return grad.cpu().numpy(), dx.cpu().numpy()


def test_noalloc_backward_matches_the_allocating_one(dev):  # noqa: F811
    for k, (name, mk, B, dtype) in enumerate(CASES):
        print(f"case {name}", flush=True)
        net = mk()
        st = hp.Stage(to_layers(net), B, net.H, net.W, net.C, dtype=dtype)
        w = oracle_weights(net, 300 + k, scale_bn=True)
        xa, lab, dya = make_inputs(net, B, 301 + k, dy_std=1e-3)
        wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(dev)
        xt = torch.from_numpy(np.ascontiguousarray(xa, np.float32)).to(dev)
        lt = torch.from_numpy(lab).to(dev) if lab is not None else None
        dyt = torch.from_numpy(np.ascontiguousarray(dya, np.float32)).to(dev) \
            if dya is not None else None
        g0, dx0 = _run(st, net, B, wt, xt, lt, dyt, noalloc=False)
        g1, dx1 = _run(st, net, B, wt, xt, lt, dyt, noalloc=True)
        g2, dx2 = _run(st, net, B, wt, xt, lt, dyt, noalloc=False)   # the stage's own again
        assert np.all(np.isfinite(g0)) and np.all(np.isfinite(dx0)), name
        assert np.array_equal(g1.view(np.uint32), g0.view(np.uint32)), f"{name}: gradient"
        assert np.array_equal(dx1.view(np.uint32), dx0.view(np.uint32)), f"{name}: dx"
        assert np.array_equal(g2.view(np.uint32), g0.view(np.uint32)), f"{name}: gradient after"
        st.close()


def test_noalloc_backward_argument_errors(dev):  # noqa: F811
    net = onets.tiny(8, 8)
    st = hp.Stage(to_layers(net), 1, 8, 8, 3)
    w = torch.zeros(st.P, device=dev)
    g = torch.zeros(st.P, device=dev)
    with pytest.raises(hp.HPError) as e:            # no forward pass before it
        st.backward_noalloc(w, None, None, g)
    assert e.value.code == hp.HP_ERR_STATE
    st.close()
    L = hp.lib()
    assert L.hp_stage_backward_noalloc(None, None, None, None, None) == hp.HP_ERR_ARG
