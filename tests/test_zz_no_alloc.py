"""dif_attention_ex_static (no allocation, library-held split workspace)
against dif_attention_ex with a caller workspace, through the C ABI.

Two calls in a row on the same device, the second with a smaller input, so
the second runs over the buffer the first left behind: both must give the
same bits as dif_attention_ex (the same kernels and launch), and both cases
must exercise the key split.
"""
import math

import numpy as np
import pytest

from paper_2607_06631_amd import binding as B
from tests.gpu_util import say
from workloads import synth

pytestmark = [pytest.mark.gpu]

LOG2E = 1.4426950408889634


def _inputs(L, heads, batch, seed):
    import torch
    dh = 128
    q, k, v = synth.make_attention_inputs(L * batch, heads, dh, 2.0, 2.0, seed)
    qs = synth.bf16_round(q * np.float32(LOG2E / math.sqrt(dh)))
    w = heads * dh
    ldvt = -(-L // 64) * 64
    Qd = torch.from_numpy(qs).cuda().to(torch.bfloat16).contiguous()
    Kd = torch.from_numpy(k).cuda().to(torch.bfloat16).contiguous()
    Vt = torch.zeros((batch * w, ldvt), dtype=torch.bfloat16, device="cuda")
    vd = torch.from_numpy(v).cuda().to(torch.bfloat16)
    for b in range(batch):
        Vt[b * w:(b + 1) * w, :L] = vd[b * L:(b + 1) * L].t()
    return Qd, Kd, Vt, w, ldvt


def _splits(L, heads, batch, ncu):
    items = -(-L // 256) * heads * batch
    rem = items % ncu
    return 0 < rem and 2 * rem <= ncu and rem <= 128


@pytest.mark.parametrize("first,second", [((32760, 29, 1), (4551, 9, 2))])
def test_static_scratch_matches_caller_workspace(first, second):
    import torch
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    ws = torch.empty(B.dif_attention_split_bytes(128), dtype=torch.uint8, device="cuda")
    for i, (L, heads, batch) in enumerate((first, second)):
        assert _splits(L, heads, batch, ncu), (L, heads, batch, ncu)
        say(f"no-alloc attention call {i}: L={L} heads={heads} batch={batch}")
        Qd, Kd, Vt, w, ldvt = _inputs(L, heads, batch, seed=20 + i)
        o_ref = torch.empty((batch * L, w), dtype=torch.bfloat16, device="cuda")
        o_st = torch.full((batch * L, w), float("nan"), dtype=torch.bfloat16, device="cuda")
        B.dif_attention_ex(Qd, Kd, Vt, o_ref, batch, L, L, heads, 128, w, w, ldvt, w,
                           flags=B.DIF_ATTN_Q_PRESCALED, split_ws=ws)
        B.dif_attention_ex_static(Qd, Kd, Vt, o_st, batch, L, L, heads, 128, w, w, ldvt, w,
                                  flags=B.DIF_ATTN_Q_PRESCALED)
        torch.cuda.synchronize()
        assert torch.isfinite(o_st.float()).all().item()
        same = torch.equal(o_st, o_ref)
        say(f"  identical: {same}")
        assert same
