"""GPU check of ifq_run_stack_static, the stack driver for callers that
cannot allocate: on the same seeded stacks and inputs its output must equal
ifq_run_stack's (which allocates nothing either, but takes the caller's
workspace) bit for bit, over two calls in a row on the shared static
workspace, the second with a smaller batch."""
import numpy as np
import pytest

from oracle import stack as ostack
from workloads import get_stack

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


def _run_both(P, cfg, batch, layout, fuse):
    import torch
    params = ostack.stack_params(cfg, "plain")
    x_host = ostack.stack_x(cfg, batch)
    dev = P.DeviceStack(get_stack(cfg).layers, params, batch, code_layout=layout,
                        fuse_down=fuse, fuse_pool=fuse)
    assert P.ifq_stack_workspace_bytes(dev.stack) <= P.ifq_static_workspace_bytes()
    x = dev.upload_input(x_host)
    y_ref = dev.alloc_output()
    y_ref.fill_(0x5A)
    dev.run(x, y_ref)
    torch.cuda.synchronize()
    y = dev.alloc_output()
    y.fill_(0xA5)
    dev.run_static(x, y)
    torch.cuda.synchronize()
    return y_ref, y


@pytest.mark.parametrize("cfg,batches,layout,fuse", [
    (3, (64, 8), "b64", True),    # the benchmark's stack at full batch, then 8
    (4, (8, 2), "b64", True),     # the detector stack (8-bit first layer, int32 head)
    (1, (32, 5), "u2", False),    # AlexNet body, separate pools, NHWC packed codes
])
def test_static_workspace_matches_caller_workspace(P, cfg, batches, layout, fuse):
    print("run_stack_static: config %d, batches %s, layout %s" % (cfg, batches, layout),
          flush=True)
    for batch in batches:
        y_ref, y = _run_both(P, cfg, batch, layout, fuse)
        assert y.numel() == y_ref.numel() and y.numel() > 0
        assert np.array_equal(y.cpu().numpy(), y_ref.cpu().numpy()), (cfg, batch)


def test_static_rejects_a_stack_larger_than_its_workspace(P):
    # the ResNet-shaped stack at batch 64 in byte-per-code layout needs about
    # 133 MiB of slots: refused before any launch, the output untouched
    import torch
    params = ostack.stack_params(3, "plain")
    dev = P.DeviceStack(get_stack(3).layers, params, 64, code_layout="i8")
    need = P.ifq_stack_workspace_bytes(dev.stack)
    assert need > P.ifq_static_workspace_bytes()
    x = dev.alloc_input()
    y = dev.alloc_output()
    y.fill_(7)
    with pytest.raises(P.IfqError) as e:
        dev.run_static(x, y)
    assert e.value.status == -4 and "static workspace" in str(e.value)
    torch.cuda.synchronize()
    assert bool((y == 7).all())
