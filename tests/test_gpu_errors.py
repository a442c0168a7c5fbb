"""Failure handling on the GPU: a plan that cannot get its device memory is refused with DR_ENOMEM,
frees what it had taken, and the library works again once memory is back."""
import pytest
import torch

from paper_2607_22614_amd import dr, workloads
from tests.gpu_helpers import require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _fill_device_memory():
    """Device memory taken in shrinking blocks until no block of 1 MiB is left."""
    hogs = []
    for block in (1 << 30, 64 << 20, 4 << 20, 1 << 20):
        while True:
            try:
                hogs.append(torch.empty(block, dtype=torch.uint8, device="cuda"))
            except torch.OutOfMemoryError:
                break
    return hogs


def test_out_of_device_memory_is_dr_enomem():
    wl = workloads.EIGHT_B  # its plan holds about 51 MB of device tables
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    hogs = _fill_device_memory()
    say("plan creation with device memory full:", sum(h.numel() for h in hogs) >> 20, "MiB taken")
    try:
        with pytest.raises(dr.DrError) as e:
            dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
        assert e.value.code == dr.DR_ENOMEM and "hipMalloc" in str(e.value)
    finally:
        del hogs
        torch.cuda.empty_cache()
    # the failure was reported by the library alone: the caller's own HIP work goes on (the
    # runtime's last error was consumed, so a framework that checks it after its launches does
    # not raise on it)
    x = torch.ones(1 << 26, device="cuda")
    assert int(x.sum().item()) == 1 << 26
    plan = dr.dr_plan_create(wl.model, wl.train_shards, wl.tp, wl.chunk_bytes)
    assert dr.dr_plan_get_info(plan)["device"] == torch.cuda.current_device()
    plan.close()
