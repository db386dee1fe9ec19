"""o5_policy_sample_static (no workspace, static device scratch) against
o5_policy_sample on the same inputs: two calls in a row, the second with a
smaller batch (and a unit-selection head, so it uses a different part of
the scratch), must give bitwise the same actions, log-probabilities and
values; a shape beyond the static scratch is rejected with O5_E_SHAPE and
leaves its outputs untouched."""
import numpy as np
import pytest
import torch

from paper_1912_06680_amd import o5
from tests.gpu_util import banner, dev, dev_bf16, dev_f32, need_gpu, workspace

pytestmark = pytest.mark.gpu


def _case(B, H, heads, seed, unit_d=0):
    rng = np.random.Generator(np.random.PCG64(seed))
    A1 = sum(heads) + 1
    h = np.tanh(rng.standard_normal((B, H), dtype=np.float32))
    Wp = ((rng.random((A1, H), dtype=np.float32) * 2 - 1) * 4 / np.sqrt(H)).astype(np.float32)
    bp = ((rng.random(A1, dtype=np.float32) * 2 - 1) / np.sqrt(H)).astype(np.float32)
    avail = (rng.random((B, A1 - 1)) < 0.8).astype(np.uint8)
    out = dict(h=dev_bf16(h), Wp=dev_bf16(Wp), bp=dev_f32(bp), avail=dev(avail), unit=None, keep=[])
    if unit_d:
        nk = heads[1]
        Wq = dev_bf16(((rng.random((unit_d, H), dtype=np.float32) * 2 - 1) / np.sqrt(H)).astype(np.float32))
        bq = dev_f32(np.zeros(unit_d, np.float32))
        E = dev_bf16(rng.standard_normal((B, nk, unit_d), dtype=np.float32) / np.sqrt(unit_d))
        out["unit"] = o5.unit_head(1, unit_d, Wq, bq, E)
        out["keep"] = [Wq, bq, E]
    return out


def _outs(B, K):
    return (torch.full((B, K), 7, dtype=torch.int32, device="cuda"),
            torch.full((B,), 1234.5, dtype=torch.float32, device="cuda"),
            torch.full((B,), 1234.5, dtype=torch.float32, device="cuda"))


def test_static_scratch_sampler_matches_workspace_sampler():
    need_gpu()
    dt = o5.O5_BF16
    for B, H, heads, seed, counter, unit_d in ((4096, 4096, (30, 8, 32, 4), 1, 3, 0),
                                                (300, 512, (30, 40, 32, 4), 2, 4, 64)):
        banner(f"static-scratch sampler B={B} H={H} heads={heads} unit_d={unit_d}")
        c = _case(B, H, heads, seed, unit_d)
        K = len(heads)
        ref = _outs(B, K)
        ws = workspace(o5.o5_policy_sample_workspace_bytes(dt, B, H, heads, unit=c["unit"]))
        o5.o5_policy_sample(dt, B, H, heads, c["h"], c["Wp"], c["bp"], 11, counter, *ref, ws, avail=c["avail"],
                            unit=c["unit"])
        got = _outs(B, K)
        o5.o5_policy_sample_static(dt, B, H, heads, c["h"], c["Wp"], c["bp"], 11, counter, *got, avail=c["avail"],
                                   unit=c["unit"])
        torch.cuda.synchronize()
        for name, a, b in zip(("act", "logp", "value"), got, ref):
            assert torch.equal(a, b), name
        assert (ref[0] >= -1).all() and torch.isfinite(ref[2]).all()
        print(f"    B={B}: act, logp, value bitwise equal", flush=True)


def test_static_scratch_sampler_rejects_shapes_beyond_its_scratch():
    need_gpu()
    dt = o5.O5_BF16
    heads = (30, 8, 32, 4)
    B, H = 16384, 4096
    banner(f"static-scratch sampler rejects B={B} H={H}")
    assert o5.o5_policy_sample_workspace_bytes(dt, B, H, heads) > (16 << 20)
    h = torch.zeros((B, H), dtype=torch.bfloat16, device="cuda")
    Wp = torch.zeros((75, H), dtype=torch.bfloat16, device="cuda")
    bp = torch.zeros(75, dtype=torch.float32, device="cuda")
    outs = _outs(B, len(heads))
    with pytest.raises(o5.O5Error) as e:
        o5.o5_policy_sample_static(dt, B, H, heads, h, Wp, bp, 1, 0, *outs)
    assert e.value.status == 2 and "static buffer" in str(e.value)
    torch.cuda.synchronize()
    assert (outs[0] == 7).all() and (outs[1] == 1234.5).all() and (outs[2] == 1234.5).all()
