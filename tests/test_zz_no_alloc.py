"""The allocation-free decode entry point (glide_decode_step_noalloc) against
glide_decode_step with a caller's workspace: the same kernels, so outputs and
states must agree bit for bit.  Two calls in a row on the library's fixed
scratch, the second with a smaller input (fewer layers, sequences and heads,
a narrower head): both split their windows over several workgroups, so both
go through the scratch records, and the second runs on what the first left
there."""
import pytest
import torch

from paper_2607_24788_amd import glide

pytestmark = pytest.mark.gpu

CASES = [
    # windows, batch, Hq, Hkv, d, Df, dtype, prefill lengths, decode steps
    ([0, 300, 2000], 2, 16, 2, 128, 128, torch.bfloat16, [700, 1500], 3),
    ([5, 400], 1, 4, 1, 64, 64, torch.float32, [450], 2),
]


def _run(case, noalloc):
    windows, B, Hq, Hkv, d, Df, dtype, lens, steps = case
    L = len(windows)
    g = glide.Glide(L, B, Hq, Hkv, d, Df, windows, dtype=dtype)
    gen = torch.Generator().manual_seed(31 + L)
    n = max(lens) + steps
    q = (torch.randn((L, B, n, Hq, d), generator=gen) * d ** -0.5).to(dtype)
    k = (torch.randn((L, B, n, Hkv, d), generator=gen) * d ** -0.5).to(dtype)
    v = (torch.randn((L, B, n, Hkv, d), generator=gen) * d ** -0.5).to(dtype)
    wf = (torch.randn((L, d, Df), generator=gen) * d ** -0.5).to(dtype).cuda()
    cu = [0]
    for x in lens:
        cu.append(cu[-1] + x)
    pack = lambda x: torch.cat([x[:, b, :lens[b]] for b in range(B)], 1).contiguous().cuda()
    st = g.new_state()
    g.state_init(st)
    ws = g.new_workspace(cu[-1])
    assert g.workspace_bytes(0) > 256, "the case must split windows"
    pout = torch.empty((L, cu[-1], Hq, d), dtype=dtype, device="cuda")
    g.prefill(st, wf, pack(q), pack(k), pack(v), cu, pout, ws)
    outs = []
    for s in range(steps):
        sel = lambda x: torch.stack([x[:, b, lens[b] + s] for b in range(B)], 1).contiguous().cuda()
        o = torch.full((L, B, Hq, d), float("nan"), dtype=dtype, device="cuda")
        if noalloc:
            g.decode_step_noalloc(st, wf, sel(q), sel(k), sel(v), o)
        else:
            g.decode_step(st, wf, sel(q), sel(k), sel(v), o, ws)
        outs.append(o)
    torch.cuda.synchronize()
    return torch.stack(outs).cpu(), st.cpu()


def test_noalloc_decode_equals_workspace_decode_twice_in_a_row():
    for i, case in enumerate(CASES):
        print(f"no-alloc decode case {i}: windows {case[0]}, batch {case[1]}, d {case[4]}", flush=True)
        want_o, want_st = _run(case, noalloc=False)
        got_o, got_st = _run(case, noalloc=True)
        assert torch.isfinite(got_o.float()).all(), f"case {i}: non-finite output"
        assert torch.equal(got_o, want_o), f"case {i}: outputs differ"
        assert torch.equal(got_st, want_st), f"case {i}: states differ"
