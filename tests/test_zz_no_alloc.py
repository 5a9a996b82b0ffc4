"""ld_attn_bwd_noalloc (the attention backward with its delta rows in the
library's fixed scratch array, for callers that cannot allocate) against
ld_attn_bwd with a caller workspace, through the C ABI (needs a GPU).

Two calls in a row on the same GPU, the second with a smaller input, so the
second runs over what the first left in the shared array; both must equal
the workspace entry point's results bit for bit (same kernels, same
arithmetic; only where delta lives differs).  Requests beyond the array are
refused before anything is launched."""
import pytest
import torch

import paper_2609_05275_amd as ld
from tests.gpu_util import DEV

pytestmark = pytest.mark.gpu

TD = {"bf16": torch.bfloat16, "f32": torch.float32}


def _inputs(dt, n, S, H, dh, seed):
    d = H * dh
    g = torch.Generator().manual_seed(seed)
    qkv = torch.randn(n * S, 3 * d, generator=g).to(TD[dt]).to(DEV)
    go = torch.randn(n * S, d, generator=g).to(TD[dt]).to(DEV)
    o = torch.empty(n * S, d, dtype=TD[dt], device=DEV)
    lse = torch.empty(n, H, S, dtype=torch.float32, device=DEV)
    return qkv, go, o, lse


def _both(dt, n, S, H, dh, alibi, seed):
    d = H * dh
    print(f"[no-alloc] {dt} n={n} S={S} H={H} dh={dh} alibi={alibi}", flush=True)
    qkv, go, o, lse = _inputs(dt, n, S, H, dh, seed)
    ld.ld_attn_fwd(n, S, H, dh, qkv, o, lse, alibi=alibi)
    ws = torch.empty(ld.ld_attn_bwd_ws_bytes(n, S, H), dtype=torch.uint8, device=DEV)
    want = torch.full((n * S, 3 * d), 5.0, dtype=TD[dt], device=DEV)
    ld.ld_attn_bwd(n, S, H, dh, qkv, o, lse, go, want, ws, alibi=alibi)
    got = torch.full((n * S, 3 * d), -5.0, dtype=TD[dt], device=DEV)
    ld.ld_attn_bwd_noalloc(n, S, H, dh, qkv, o, lse, go, got, alibi=alibi)
    torch.cuda.synchronize()
    assert torch.isfinite(want.float()).all()
    assert torch.equal(got, want)


@pytest.mark.parametrize("dt,first,second", [
    ("bf16", (4, 512, 4, 128, 1), (2, 256, 2, 64, 0)),
    ("bf16", (8, 2048, 16, 128, 0), (3, 192, 2, 64, 1)),    # the 1B shape, then a ragged small one
    ("f32", (3, 96, 4, 16, 0), (2, 32, 2, 64, 1)),
])
def test_noalloc_matches_workspace_entry_point(dt, first, second):
    _both(dt, *first, seed=1)
    _both(dt, *second, seed=2)


def test_noalloc_refuses_beyond_the_fixed_scratch():
    n, S, H, dh = 64, 2048, 32, 64        # 2^22 delta rows > 2^21
    qkv = torch.zeros(64, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ld.LdError) as e:
        ld.ld_attn_bwd_noalloc(n, S, H, dh, qkv, qkv, qkv.float(), qkv, qkv)
    assert e.value.status == 3              # LD_E_UNSUPPORTED, nothing launched
    assert "fixed scratch" in str(e.value)
