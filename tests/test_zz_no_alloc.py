"""The selection entry point that allocates nothing (tp_combine_select_topk_static), through
the C ABI on the GPU: its kept sets equal tp_combine_select_topk's (with a workspace) bit for
bit, on two calls in a row, the second with a smaller input, so the static buffer holds the
first call's larger contents when the second runs."""
import numpy as np
import pytest
import torch

from paper_2608_03276_amd import binding as B

import parity_util as pu

pytestmark = pytest.mark.gpu


def _case(rng, L, Hkv, lens, ties):
    n = L * Hkv * sum(lens)
    s_key = rng.random(n, dtype=np.float32)
    scales = rng.random(n, dtype=np.float32)
    if ties:  # many equal combined scores, so the tie rule decides part of each kept set
        s_key = np.round(s_key * 8) / 8
        scales = np.ones(n, dtype=np.float32)
    return torch.from_numpy(s_key).cuda(), torch.from_numpy(scales).cuda()


@pytest.mark.parametrize("rule", [B.TP_COMBINE_MUL, B.TP_COMBINE_NORM_ADD])
def test_static_selection_matches_workspace_selection(gpu_lib, rule):
    rng = np.random.default_rng(77)
    # first call: 4 segments over a ragged batch (close to the buffer's size), then a smaller one
    for L, Hkv, lens, ratio, budget, ties in [(2, 2, [2000000, 1000000, 7], 0.1, 0, False),
                                              (1, 2, [5000, 1, 333], 0.0, 700, True)]:
        pu.log(f"static selection rule={rule} L={L} Hkv={Hkv} lens={lens}")
        d = B.dims(L, Hkv, Hkv, 64)
        bt = B.Batch(np.concatenate([[0], np.cumsum(lens)]).tolist())
        assert B.tp_workspace_size(B.TP_FN_COMBINE_SELECT_TOPK, d, bt) <= B.TP_STATIC_SCRATCH_BYTES
        ko = B.kept_offsets_for(bt, ratio, budget)
        s_key, scales = _case(rng, L, Hkv, lens, ties)
        kept_ref = torch.full((L * Hkv * ko[-1],), -1, dtype=torch.int32, device="cuda")
        kept = torch.full_like(kept_ref, -2)
        ws = torch.empty(B.tp_workspace_size(B.TP_FN_COMBINE_SELECT_TOPK, d, bt), dtype=torch.uint8, device="cuda")
        B.tp_combine_select_topk(d, bt, s_key, scales, rule, ratio, budget, ko, kept_ref, None, ws)
        B.tp_combine_select_topk_static(d, bt, s_key, scales, rule, ratio, budget, ko, kept)
        torch.cuda.synchronize()
        assert torch.equal(kept, kept_ref)
        assert int(kept_ref.min()) >= 0
