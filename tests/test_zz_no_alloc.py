"""The no-allocation variant of the layer (clearmoe_ffn_forward_noalloc),
called through the C ABI, against clearmoe_ffn_forward with a caller
workspace: the same kernels run, so y, the expert indices and the gates must
agree bit for bit.  Each case makes two calls in a row on the library's one
scratch array, the second with fewer tokens, so that the second call starts
from the first call's leftovers (the split counters and partials are cleared
by the call itself)."""
import numpy as np
import pytest
import torch

from paper_2606_28516_amd import clearmoe as cm
from paper_2606_28516_amd import synth

from parity_util import layer_to_device

pytestmark = pytest.mark.gpu

# (name, first T, second T, D, H, E, k, r, q, dtype): the fused top-1 kernel
# (the second call takes its hidden split, which keeps partials and arrival
# counters in scratch), the float32 top-1 GEMM chain (split-K counters), and
# a top-2 GEMM chain.
CASES = [
    ("fused_top1", 12608, 3000, 384, 1536, 8, 1, 128, 32, "bf16"),
    ("chain_top1_f32", 1576, 700, 192, 768, 4, 1, 64, 16, "f32"),
    ("chain_top2_bf16", 2000, 517, 128, 256, 6, 2, 32, 16, "bf16"),
]


def _layer(T, D, H, E, k, r, q, dt, seed):
    cfg = synth.LayerConfig("noalloc", T=T, D=D, H=H, E=E, k=k, r=r, q=q, dtype=dt, seed=seed,
                            residual="random", n_cal=3000)
    return synth.make_layer(cfg)


@pytest.mark.parametrize("name,T0,T1,D,H,E,k,r,q,dt", CASES)
def test_noalloc_matches_workspace_entry_point(name, T0, T1, D, H, E, k, r, q, dt):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    for i, T in enumerate((T0, T1)):
        print(f"case {name} call {i}: T={T}", flush=True)
        L = _layer(T, D, H, E, k, r, q, dt, seed=T + i)
        d = layer_to_device(L)
        args = [d[n] for n in ("x", "W1", "b1", "US", "Vt", "b2", "P", "Q", "Wg", "bg")]
        idx_a = torch.empty((T, k), dtype=torch.int32, device="cuda")
        gate_a = torch.empty((T, k), dtype=torch.float32, device="cuda")
        y_a = cm.ffn_forward_noalloc(*args, k, idx_out=idx_a, gate_out=gate_a)
        idx_b = torch.empty_like(idx_a)
        gate_b = torch.empty_like(gate_a)
        y_b = cm.ffn_forward(*args, k, idx_out=idx_b, gate_out=gate_b)
        torch.cuda.synchronize()
        assert torch.equal(idx_a, idx_b)
        assert torch.equal(gate_a, gate_b)
        ya, yb = cm.to_stored(y_a), cm.to_stored(y_b)
        assert np.array_equal(ya, yb), f"{int((ya != yb).sum())} elements differ"
