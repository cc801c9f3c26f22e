"""The allocation-free NMSE entry point (saf3r_nmse_noalloc) against
saf3r_nmse with a caller workspace: the same kernels and reduction order, so
the same float64 bits, on consecutive calls whose sizes shrink (the
library's per-GPU array keeps the previous call's partial sums, which the
next call must not read)."""
import pytest

pytestmark = pytest.mark.gpu


def test_nmse_noalloc_matches_the_workspace_entry(gpu_lib):
    import torch

    import paper_2607_03612_amd as P

    g = torch.Generator(device="cuda").manual_seed(2607)
    # the most heads the array holds, a benchmark-sized layer, then smaller ones
    cases = [(256, 3, 87, torch.bfloat16), (16, 7, 1374, torch.bfloat16), (5, 2, 261, torch.float32),
             (3, 1, 40, torch.bfloat16)]
    for heads, frames, T, dtype in cases:
        n = frames * T
        print(f"[no-alloc] heads {heads} N {n} {dtype}", flush=True)
        full = torch.randn((heads, n, 64), generator=g, device="cuda").to(dtype)
        noise = torch.randn((heads, n, 64), generator=g, device="cuda")
        sparse = (full.float() + 0.05 * noise).to(dtype)
        want = P.nmse(full, sparse, frames, T)
        got = torch.full((heads,), float("nan"), dtype=torch.float64, device="cuda")
        P.nmse_noalloc(full, sparse, frames, T, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want), (heads, n, (got - want).abs().max().item())
        assert bool(torch.isfinite(got).all()) and bool((got > 0).all())
