"""Plan upload and the plan's host image.

pfx_plan_upload copies the plan's host image (pageable memory) into the
device workspace with an asynchronous copy on the given stream, and a
destroyed plan's image is reused by the next plan built on the thread.  The
copy must therefore have read the image by the time the upload returns.
Here the upload is queued behind attention work on its stream, the plan is
destroyed at once, and a plan of the same size over other pages is built
over the same image and uploaded; the first workspace must hold exactly the
first plan's image, byte for byte, and the two images must differ."""

import gc

import pytest
import torch

from paper_2608_25523_amd import binding as B
from paper_2608_25523_amd import runner as RN
from paper_2608_25523_amd import workloads as W

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu-test] {msg}", flush=True)


@pytest.mark.timeout(300)
def test_plan_destroyed_right_after_upload_keeps_its_workspace():
    b = W.config_batch(2)
    other = W.replicas(b, 2, 91)[1]              # same lengths and agents, other pages
    announce("plan upload: config-2 decode plan uploaded behind attention work, destroyed, image reused")
    ds = RN.DeviceStep(b, W.host_values_fast(b, 9), poison=False)
    nbytes = ds.plan.workspace_bytes()

    ws_ref = torch.zeros(nbytes + 256, dtype=torch.uint8, device="cuda")
    ws_a = torch.zeros_like(ws_ref)
    ws_b = torch.zeros_like(ws_ref)
    ref = B.plan_from_batch(ds.pool, b, B.PFX_MODE_DECODE).upload(workspace=ws_ref)
    torch.cuda.synchronize()
    del ref
    gc.collect()

    for _ in range(20):                          # work queued ahead of the uploads
        ds.attention()
    a = B.plan_from_batch(ds.pool, b, B.PFX_MODE_DECODE).upload(workspace=ws_a)
    a.workspace = None
    del a
    gc.collect()                                 # its image is now the spare
    c = B.plan_from_batch(ds.pool, other, B.PFX_MODE_DECODE)
    assert c.workspace_bytes() == nbytes
    c.upload(workspace=ws_b)
    torch.cuda.synchronize()
    B.pfx_sync_check()

    assert torch.equal(ws_a, ws_ref), "the destroyed plan's workspace differs from its image"
    assert not torch.equal(ws_b, ws_ref), "the second plan should differ (other pages)"
    del c
    announce("plan upload: workspace holds the destroyed plan's image")
