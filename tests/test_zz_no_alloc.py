"""cnn_fwd_plan_static: the same kernels as cnn_fwd_plan_ws, with the
library's static device scratch as the workspace (for callers that cannot
allocate).  Compared with cnn_fwd_plan_ws on the same plan, and with the
oracle, on two calls in a row per case, the second on a smaller problem
(the scratch keeps the first call's contents)."""
import numpy as np
import pytest

import oracle
from paper_2105_13480_amd import cnn, inputs

from gpu_helpers import out_tensor, say, to_gpu, to_host64

pytestmark = pytest.mark.gpu

MODES = {"f32": cnn.CNN_F32, "bf16": cnn.CNN_BF16, "bf16_obf16": cnn.CNN_BF16_OBF16}

# (first problem, second smaller problem, mode, kernel, tk, tp, tc): plans
# that need a workspace (channel-split partial Outs, a repacked Ker)
CASES = [
    ((1, 512, 512, 7, 7, 3, 3, 1, 1), (1, 256, 128, 7, 7, 3, 3, 1, 1), "bf16", cnn.K_SPLITC, 32, 256, 32),
    ((1, 16, 16, 16, 16, 3, 3, 1, 1), (1, 16, 8, 9, 5, 3, 3, 1, 1), "f32", cnn.K_SPLITC, 64, 64, 8),
    ((2, 32, 300, 7, 28, 3, 3, 2, 2), (1, 16, 64, 7, 28, 3, 3, 2, 2), "bf16_obf16", cnn.K_SROWS, 256, 7 * 28, 16),
    ((1, 512, 512, 7, 7, 3, 3, 1, 1), (1, 96, 70, 7, 7, 3, 3, 1, 1), "bf16_obf16", cnn.K_SPLITC, 32, 64, 32),
]


def _ints(dims, mode, seed):
    return inputs.make_arrays(*dims, "f32" if mode == "f32" else "bf16", seed_in=seed,
                              seed_ker=seed + 1, in_dist=("int", -2, 2), ker_dist=("int", -2, 2))


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"k{c[3]}_{c[2]}")
def test_static_scratch_matches_caller_workspace(case):
    import torch
    first, second, mode, kernel, tk, tp, tc = case
    dt = MODES[mode]
    for i, dims in enumerate((first, second)):
        Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
        pl = cnn.plan_tiles(cnn.problem(*dims), dt, kernel, tk, tp, tc)
        assert 0 < pl.ws_bytes <= cnn.STATIC_SCRATCH_BYTES
        In, Ker = _ints(dims, mode, seed=100 * i + kernel)
        dIn, dKer = to_gpu(In), to_gpu(Ker)
        ref = out_tensor(Nb, Nk, Nw, Nh, mode)
        ws = torch.empty(pl.ws_bytes, dtype=torch.uint8, device="cuda")
        if i == 1:  # the caller's workspace of the first call is no longer needed
            torch.cuda.synchronize()
        say(f"[static] call {i + 1} dims={dims} mode={mode} kernel={kernel} v{pl.variant} "
            f"ws={pl.ws_bytes}: cnn_fwd_plan_ws")
        cnn.fwd_plan_ws(dIn, dKer, ref, pl, ws, sw, sh)
        torch.cuda.synchronize()
        got = out_tensor(Nb, Nk, Nw, Nh, mode)
        say(f"[static] call {i + 1}: cnn_fwd_plan_static")
        cnn.fwd_plan_static(dIn, dKer, got, pl, sw, sh)
        torch.cuda.synchronize()
        # The first call on a device loads the scratch (static device data of
        # the library, held until the process ends); later calls allocate
        # nothing.
        free1, _ = torch.cuda.mem_get_info()
        if i == 0:
            free_after_first = free1
        else:
            assert free1 == free_after_first
        g, r = to_host64(got), to_host64(ref)
        assert np.array_equal(g, r)
        want = oracle.conv(In, Ker, sw, sh)
        if mode == "bf16_obf16":
            want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
        assert np.array_equal(g, want)
