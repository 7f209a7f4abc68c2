"""kan_layer_forward_noalloc (packed weights in the library's fixed per-device
scratch array, nothing allocated) against kan_layer_forward (packed weights in
a caller workspace), both through the raw C entry points: two calls in a row,
the second on a smaller layer, each bit-identical to the workspace entry point
and within the layer tolerance of the float64 oracle."""
import numpy as np
import pytest

import oracle
from paper_2609_01956_amd import binding as kb
from paper_2609_01956_amd import workloads as wl
from gpu_common import (BF16_LAYER_TOL, F32_LAYER_TOL, device, normwise, say, to_dev,
                        to_host64, torch)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype_name", ["f32", "bf16"])
def test_noalloc_matches_workspace_entry_point(dtype_name):
    dt = torch.float32 if dtype_name == "f32" else torch.bfloat16
    code = kb.KAN_F32 if dtype_name == "f32" else kb.KAN_BF16
    tol = F32_LAYER_TOL if dtype_name == "f32" else BF16_LAYER_TOL
    stream = int(torch.cuda.current_stream().cuda_stream)
    cap = kb.KAN_NOALLOC_SCRATCH_BYTES
    # a layer of the 784-wide MLP input at a reduced batch, then smaller ones:
    # the second splits its contraction with the partial sums in the scratch
    # array too; last a narrow layer at a batch where fp32 runs the vector-ALU
    # kernel
    for B, n_in, n_out, G in [(1000, 784, 256, 10), (64, 784, 64, 5), (300, 17, 40, 7),
                              (16400, 33, 10, 10)]:
        x, C, Wb = wl.make_layer(wl.LayerShape(B, n_in, n_out, G, off_grid_frac=0.1),
                                 seed=B + n_in)
        if dtype_name == "bf16":
            x, C, Wb = (wl.round_to_bf16_f32(a) for a in (x, C, Wb))
        xt, Ct, Wt = to_dev(x, dt), to_dev(C, dt), to_dev(Wb, dt)
        g = kb.make_grid(G)
        y_na = torch.full((B, n_out), float("nan"), dtype=dt, device=device())
        y_ws = torch.empty((B, n_out), dtype=dt, device=device())
        st, need = kb.kan_layer_forward_workspace_bytes(g, code, B, n_in, n_out)
        packed = kb.kan_layer_packed_bytes(g, code, n_in, n_out)[1]
        assert st == kb.KAN_OK and packed <= cap
        st, plan = kb.kan_layer_plan(g, code, B, n_in, n_out)
        if (B, n_in) == (64, 784):
            assert plan[5] > 1 and packed < need <= cap
        if B == 16400 and dtype_name == "f32":
            assert plan[:4] == (0, 4, 4, 1)
        # the workspace entry point gets the bytes the scratch array offers:
        # where the partial sums do not fit there, both run unsplit
        ws = torch.empty(min(need, cap), dtype=torch.uint8, device=device())
        say(f"noalloc {dtype_name} B={B} in={n_in} out={n_out} G={G} splits={plan[5]} "
            f"need={need}")
        assert kb.kan_layer_forward_noalloc(g, code, B, n_in, n_out, xt.data_ptr(), Ct.data_ptr(),
                                            Wt.data_ptr(), y_na.data_ptr(), stream) == kb.KAN_OK
        assert kb.kan_layer_forward(g, code, B, n_in, n_out, xt.data_ptr(), Ct.data_ptr(),
                                    Wt.data_ptr(), ws.data_ptr(), ws.numel(), y_ws.data_ptr(),
                                    stream) == kb.KAN_OK
        torch.cuda.synchronize()
        assert torch.equal(y_na, y_ws)
        ref = oracle.layer(x, C, Wb, G)
        if dtype_name == "bf16":
            ref = oracle.round_bf16(ref)
        assert normwise(to_host64(y_na), ref) <= tol
