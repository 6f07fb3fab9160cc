"""The allocation-free KV generation entry point (adept_kv_generate_noalloc)
against adept_kv_generate with a caller workspace: same kernels, so the
caches must be identical bit for bit.  Two calls in a row, the second with a
smaller input, so the second reads none of the first call's scratch state;
and a size above the fixed scratch is rejected before anything runs."""
import numpy as np
import pytest
import torch

import adept_inputs as ai
from paper_2601_03700_amd import binding as B

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(N, D, H, hd, n_tok, n_rows, seed):
    Dq = H * hd
    g = torch.Generator(device=DEV).manual_seed(seed)
    s = torch.randn((n_tok, D), generator=g, device=DEV).to(torch.bfloat16)
    w = (0.02 * torch.randn((N, 2 * Dq, D), generator=g, device=DEV)).to(torch.bfloat16)
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(n_tok, n_rows, replace=False)).astype(np.int32)
    el = rng.integers(0, N, n_tok).astype(np.int32)
    pos = rng.integers(0, 512, n_tok).astype(np.int32)
    slot = rng.permutation(n_tok + 5)[:n_tok].astype(np.int32)
    t = lambda x: torch.from_numpy(x).to(DEV)
    return s, w, t(rows), t(el), t(pos), t(slot)


def _run(noalloc, N, D, H, hd, s, w, rows, el, pos, slot, n_slots, cos, sin):
    kc = torch.full((N, n_slots, H, hd), float("nan"), dtype=torch.bfloat16, device=DEV)
    vc = torch.full_like(kc, float("nan"))
    n = torch.tensor([rows.numel()], dtype=torch.int32, device=DEV)
    Dq = H * hd
    if noalloc:
        B.kv_generate_noalloc(N, D, H, hd, 1e-6, s, rows, n, rows.numel(), el, slot, pos, w,
                              2 * Dq * D, None, cos, sin, kc, vc, n_slots)
    else:
        ws = torch.empty(B.kv_generate_workspace_bytes(N, rows.numel()), dtype=torch.uint8,
                         device=DEV)
        B.kv_generate(N, D, H, hd, 1e-6, s, rows, n, rows.numel(), el, slot, pos, w, 2 * Dq * D,
                      None, cos, sin, kc, vc, n_slots, ws)
    torch.cuda.synchronize()
    return kc, vc


def test_kv_generate_noalloc_matches_workspace_call():
    H, hd = 4, 128
    cos = torch.empty((512, hd // 2), dtype=torch.float32, device=DEV)
    sin = torch.empty_like(cos)
    B.rope_table(512, hd, 10000.0, cos, sin)
    for N, D, n_tok, n_rows, seed in ((8, 512, 1500, 1300, 1), (5, 256, 400, 77, 2)):
        print(f"noalloc kv_generate N={N} D={D} rows={n_rows}", flush=True)
        s, w, rows, el, pos, slot = _case(N, D, H, hd, n_tok, n_rows, seed)
        ref = _run(False, N, D, H, hd, s, w, rows, el, pos, slot, n_tok + 5, cos, sin)
        got = _run(True, N, D, H, hd, s, w, rows, el, pos, slot, n_tok + 5, cos, sin)
        for a, b in zip(got, ref):
            assert torch.equal(torch.isnan(a), torch.isnan(b))
            assert torch.equal(torch.nan_to_num(a), torch.nan_to_num(b))
        assert (~torch.isnan(got[0])).any()
    # beyond the fixed scratch: rejected on the host, nothing enqueued
    big = 1 << 20
    with pytest.raises(B.AdeptError, match="scratch"):
        B.kv_generate_noalloc(32, 256, H, hd, 1e-6, s, rows, torch.tensor([1], dtype=torch.int32,
                              device=DEV), big, el, slot, pos, w, 2 * H * hd * 256, None, cos,
                              sin, got[0], got[1], 1)
