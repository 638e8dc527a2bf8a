"""numbat_conv_fwd_noalloc (static device scratch instead of a workspace) against
numbat_conv_fwd on the same inputs: equal output and batch statistics (the same kernels
run, so bit for bit), on two calls in a row, the second with a smaller problem (the scratch
keeps the first call's partials), and without statistics."""
import pytest

from parity import Inputs
from paper_2609_10632_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    from paper_2609_10632_amd import blocks
    from paper_2609_10632_amd import numbat as nb

# n, h, ci, co, k, s: a 40x40 3x3 layer, then a smaller 1x1 and a stride-2 layer
CASES = [(4, 40, 192, 192, 3, 1), (2, 20, 96, 64, 1, 1), (1, 17, 48, 96, 3, 2)]


def run_both(case, idx):
    n, h, ci, co, k, s = case
    inp = Inputs(110, idx)
    blk = blocks.ConvBlock(n, h, h, ci, co, k, s)
    x = blocks.dev_bf16(inp.normal((n, h, h, ci), synth.T_X))
    w = blocks.dev_bf16(inp.weight(co, k, ci))
    y_ref = torch.full((n, blk.ho, blk.wo, co), float("nan"), dtype=torch.bfloat16, device="cuda")
    st_ref = torch.full((2 * co,), float("nan"), device="cuda")
    nb.numbat_conv_fwd(blk.prob, x, w, y_ref, st_ref, blocks.workspace(blk.ws_fwd))
    y = torch.full_like(y_ref, float("nan"))
    st = torch.full_like(st_ref, float("nan"))
    nb.numbat_conv_fwd_noalloc(blk.prob, x, w, y, st)
    y2 = torch.full_like(y_ref, float("nan"))
    nb.numbat_conv_fwd_noalloc(blk.prob, x, w, y2, None)
    torch.cuda.synchronize()
    print(f"noalloc case {case}", flush=True)
    assert torch.equal(y, y_ref), case
    assert torch.equal(st, st_ref), case
    assert torch.equal(y2, y_ref), case


def test_noalloc_forward_matches_workspace_forward():
    for i, c in enumerate(CASES):
        run_both(c, i)
