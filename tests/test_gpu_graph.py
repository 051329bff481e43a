"""HIP graph capture of whole layer steps: a step recorded once (MoELayer.capture) and replayed gives,
on every replay, bitwise the buffers of an eager step.  Before each replay the layer's buffers are
poisoned and unrelated eager work runs, with synchronizations between the replays, so a replay that
skipped, reordered or replayed stale work (a memset node, a workspace not cleared) would show."""
import sys

import pytest
import torch

from paper_2606_26453_amd import layer as L, workloads as W
from tests.gpu_util import gpu_available, poison_

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]
DEV = "cuda:0"
SCRATCH = ("workspace", "router_ws", "aux_ws", "d_act", "d_act_sh")   # scratch, or not written (fused)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _written(lay, k):
    """The part of buffer k a step writes.  Token-major MX operands of the weight gradient span
    columns up to a bound on the padded token count; a step writes (and the products read) only the
    first p[G] of them, p the prefix of the group counts rounded up to 128."""
    v = lay.buf[k]
    if k.endswith("_qt") or k.endswith("_st"):
        cnt = torch.diff(lay.buf["offsets"].cpu().long())
        pg = int(((cnt + 127) // 128 * 128).sum())
        return v[:, :pg] if k.endswith("_qt") else v[: pg // 128]
    return v


@pytest.mark.parametrize("cfg_id,opts", [
    (0, {}),
    (2, {}),
    (0, {"router": True, "aux_alpha": 0.01}),
    (0, {"fp8_forward": True, "fp8_backward": True, "mx": True, "fp8_dw": True}),
    (2, {"combine_fused": True}),
    (5, {}),
    (2, {"full": True}),
], ids=["cfg0", "cfg2", "cfg0-router", "cfg0-mx", "cfg2-combine-fused", "cfg5-dw1", "cfg2-full"])
def test_graph_replay_bitwise(cfg_id, opts):
    import dataclasses
    opts = dict(opts)
    cfg = W.CONFIGS[cfg_id]
    if cfg_id == 2 and not opts.pop("full", False):   # full size: the shared experts' dW is split
        cfg = dataclasses.replace(cfg, T=1024)
    _say("graph replay", cfg_id, opts)
    if cfg.dw_only:
        inp = W.make_dw_inputs(cfg, 0, DEV)
        lay = L.DWOnly(cfg, inp)
    else:
        inp = W.make_inputs(cfg, 0, DEV)
        lay = L.MoELayer(cfg, inp, **opts)
    lay.step()
    lay.step()
    torch.cuda.synchronize()
    ref = {k: _written(lay, k).clone() for k in lay.buf if k not in SCRATCH}
    lay.capture()
    torch.cuda.synchronize()
    other = torch.randn((512, 512), device=DEV)
    for rep in range(3):
        for k, v in lay.buf.items():
            poison_(v)
        other = torch.tanh(other @ other.t() * 1e-3)          # unrelated eager work between replays
        torch.cuda.synchronize()
        lay.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(v.view(torch.uint8), _written(lay, k).view(torch.uint8)), (rep, k)
