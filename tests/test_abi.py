"""C-ABI checks that need no GPU: the library loads, exports every function
include/layerdrop.h declares, its host-only schedule function agrees bit for
bit with the oracle, and invalid arguments are rejected before anything is
enqueued (no call here reaches the HIP runtime)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2609_05275_amd as ld
from oracle import schedule

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "layerdrop.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return set(re.findall(r"\b(ld_[a-z0-9_]+)\s*\(", src))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 20
    lib = C.CDLL(ld.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert names == set(ld.EXPORTED)


@pytest.mark.parametrize("dist", [0, 1, 2])
@pytest.mark.parametrize("sched", [0, 1, 2])
def test_schedule_matches_oracle_bitwise(dist, sched):
    for L in (1, 2, 12, 16, 32):
        for p_max in (0.0, 0.1, 0.2, 0.5, 0.99, 1.0):
            for (t, T) in ((0, 1001), (500, 1001), (1000, 1001), (7, 1), (2000, 1001), (-3, 10)):
                for l in range(L):
                    got = ld.ld_schedule_p(dist, sched, p_max, l, L, t, T)
                    # the ABI takes p_max as float32; give the oracle that same value
                    want = schedule.rate(dist, sched, float(np.float32(p_max)), l, L, t, T)
                    assert np.float32(got) == want, (dist, sched, p_max, l, L, t, T)


def test_schedule_rejects_bad_arguments():
    for args in [(3, 0, 0.2, 0, 4, 0, 1), (0, 3, 0.2, 0, 4, 0, 1), (0, 0, 1.5, 0, 4, 0, 1),
                 (0, 0, float("nan"), 0, 4, 0, 1), (0, 0, 0.2, 4, 4, 0, 1), (0, 0, 0.2, 0, 0, 0, 1),
                 (0, 0, 0.2, 0, 4, 0, 0)]:
        with pytest.raises(ld.LdError) as e:
            ld.ld_schedule_p(*args)
        assert e.value.status == 1


def test_status_strings():
    assert ld.status_name(0) == "LD_OK"
    assert ld.status_name(4) == "LD_E_WORKSPACE"
    assert ld.status_name(99) == "LD_E_UNKNOWN"


def _cfg(**kw):
    base = dict(batch=8, seq=2048, d_model=2048, n_heads=16, d_ff=5504, dtype=ld.LD_BF16)
    base.update(kw)
    return ld.config(**base)


def test_workspace_sizes():
    c = _cfg()
    ctx = ld.ld_layer_ctx_bytes(c)
    T, d, f, H = 8 * 2048, 2048, 5504, 16
    assert ctx >= 2 * T * (8 * d + 3 * f) + 8 * T + 4 * T * H
    assert ld.ld_layer_ws_bytes(c) >= 2 * T * (7 * d + 3 * f)
    s16 = ld.ld_stack_ws_bytes(c, 16)
    assert s16 >= 16 * (ctx - 4096) + ld.ld_layer_ws_bytes(c)
    assert s16 < 288e9 / 4          # fits the GPU's HBM with room to spare
    assert ld.ld_stack_ws_bytes(_cfg(batch=4, seq=4096, d_model=4096, n_heads=32, d_ff=11008), 32) < 100e9


@pytest.mark.parametrize("kw,code", [
    (dict(n_heads=3), 2),                     # d % H != 0
    (dict(n_heads=64), 3),                    # d_head 32 unsupported in bf16
    (dict(seq=100), 2),                       # bf16 needs S % 64 == 0
    (dict(d_ff=1001), 2),
    (dict(dtype=7), 1),
    (dict(rms_eps=0.0), 1),
    (dict(batch=0), 2),
    (dict(block_kind=2), 1),
    (dict(granularity=4), 1),
    (dict(granularity=-1), 1),
])
def test_invalid_configs_rejected(kw, code):
    c = _cfg(**kw)
    assert ld.ld_layer_ctx_bytes(c) == 0
    with pytest.raises(ld.LdError) as e:
        ld.ld_gather_rows(c, 8, 8, 8, 8, stream=0)
    assert e.value.status == code


def test_invalid_p_and_pointers_rejected():
    with pytest.raises(ld.LdError) as e:
        ld.ld_masks([0.1, float("nan")], 0, 0, _Fake((2, 8)), 8, 8, stream=0)
    assert e.value.status == 1
    with pytest.raises(ld.LdError) as e:
        ld.ld_masks([1.5], 0, 0, _Fake((1, 8)), 8, 8, stream=0)
    assert e.value.status == 1
    with pytest.raises(ld.LdError) as e:
        ld.ld_masks([0.5], 0, 0, _Fake((1, 8)), None, 8, stream=0)
    assert e.value.status == 1
    c = _cfg()
    w = {k: 16 for k in ld.WEIGHT_KEYS}
    with pytest.raises(ld.LdError) as e:
        ld.ld_layer_fwd(c, w, 0, -0.1, 0, 0, 16, 16, stream=0)
    assert e.value.status == 1
    w["w_o"] = None
    with pytest.raises(ld.LdError) as e:
        ld.ld_layer_fwd(c, w, 0, 0.1, 0, 0, 16, 16, stream=0)
    assert e.value.status == 1


def test_granular_masks_reject_bad_arguments():
    with pytest.raises(ld.LdError) as e:
        ld.ld_masks_granular(4, [0.1], 0, 0, _Fake((1, 8)), 8, 8, stream=0)
    assert e.value.status == 1
    with pytest.raises(ld.LdError) as e:
        ld.ld_masks_granular(1, [0.1, -0.5], 0, 0, _Fake((2, 2, 8)), 8, 8, stream=0)
    assert e.value.status == 1


def test_sublayer_ctx_holds_two_masks():
    small = dict(batch=1000, seq=64)   # mask arrays are padded to 256 bytes
    one = ld.ld_layer_ctx_bytes(_cfg(**small))
    two = ld.ld_layer_ctx_bytes(_cfg(granularity=ld.LD_GRAN_SUBLAYER_SEQ, **small))
    assert two - one >= 1000 * 5      # a second keep row (1 B) and idx row (4 B) per sample
    assert ld.ld_layer_ctx_bytes(_cfg(granularity=ld.LD_GRAN_LAYER_BATCH, **small)) == one
    assert (ld.ld_stack_ws_bytes(_cfg(granularity=3, **small), 16)
            > ld.ld_stack_ws_bytes(_cfg(**small), 16))


def test_gemm_shape_checks():
    with pytest.raises(ld.LdError) as e:   # lda smaller than K
        ld.ld_gemm(1, 1, 64, 64, 64, _Fake((64, 64), 2), 32, _Fake((64, 64), 2), 64,
                   _Fake((64, 64), 2), 64, dtype=ld.LD_BF16, stream=0)
    assert e.value.status == 2
    with pytest.raises(ld.LdError) as e:   # bf16 K not a multiple of 8
        ld.ld_gemm(1, 1, 64, 64, 60, _Fake((64, 64), 2), 64, _Fake((64, 64), 2), 64,
                   _Fake((64, 64), 2), 64, dtype=ld.LD_BF16, stream=0)
    assert e.value.status == 2
    with pytest.raises(ld.LdError) as e:
        ld.ld_gemm(1, 1, -1, 64, 64, 8, 64, 8, 64, 8, 64, dtype=ld.LD_BF16, stream=0)
    assert e.value.status == 2


class _Fake:
    """Stands in for a device tensor in calls that must fail validation."""

    def __init__(self, shape, es=1):
        self.shape = shape
        self._es = es

    def data_ptr(self):
        return 4096

    def element_size(self):
        return self._es

    def numel(self):
        return int(np.prod(self.shape))


def test_alibi_slope_host_function():
    """ld_alibi_slope (host) against the ALiBi paper's stated slopes for 8
    and 16 heads and the oracle's rule for other counts (float32)."""
    import os
    from oracle import block
    gold = {}
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "alibi_slopes.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            h, rest = line.split(":")
            gold[int(h)] = [2.0 ** -float(e) for e in rest.split()]
    for h, want in gold.items():
        got = [ld.ld_alibi_slope(i, h) for i in range(h)]
        assert np.allclose(got, want, rtol=1e-6, atol=0), h
    for h in (3, 6, 12, 21):
        got = [ld.ld_alibi_slope(i, h) for i in range(h)]
        assert np.allclose(got, block.alibi_slopes(h), rtol=1e-6, atol=0), h
    assert ld.ld_alibi_slope(-1, 8) == 0.0 and ld.ld_alibi_slope(8, 8) == 0.0


def test_binding_rejects_host_noncontiguous_and_missized_tensors():
    """The binding refuses, before any launch, torch tensors that are on the
    host, not contiguous, of the wrong dtype or of the wrong size for the
    configuration (runs without a GPU: every case fails in Python)."""
    import torch
    c = _cfg(batch=2, seq=64, d_model=128, n_heads=2, d_ff=256)
    host = torch.zeros(2, 64, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        ld._ptr(host, "x")
    meta = torch.empty(4, 8, dtype=torch.bfloat16, device="meta")
    with pytest.raises(ValueError):
        ld._ptr(meta, "x")
    # dtype / size checks come before any pointer is taken
    with pytest.raises(ValueError, match="dtype"):
        ld._check_layer_tensors(c, acts=(("x", torch.zeros(2, 64, 128, dtype=torch.float32)),))
    with pytest.raises(ValueError, match="elements"):
        ld._check_layer_tensors(c, acts=(("x", torch.zeros(2, 63, 128, dtype=torch.bfloat16)),))
    w = {k: torch.zeros(n, dtype=torch.bfloat16) for k, n in ld._weight_numel(c).items()}
    ld._check_layer_tensors(c, w=w)
    w["w_gate_up"] = torch.zeros(256 * 128, dtype=torch.bfloat16)   # W_up only: wrong for SwiGLU
    with pytest.raises(ValueError, match="w_gate_up"):
        ld._check_layer_tensors(c, w=w)
    dw = {k: torch.zeros(n, dtype=torch.bfloat16) for k, n in ld._weight_numel(c).items()}
    with pytest.raises(ValueError, match="grad"):
        ld._check_layer_tensors(c, dw=dw)
    with pytest.raises(ValueError, match="keep_override"):
        ld.ld_layer_fwd(c, {k: 16 for k in ld.WEIGHT_KEYS}, 0, 0.1, 0, 0, 16, 16,
                        keep_override=torch.zeros(3, dtype=torch.uint8), stream=0)
    sub = _cfg(batch=2, seq=64, d_model=128, n_heads=2, d_ff=256, granularity=ld.LD_GRAN_SUBLAYER_SEQ)
    with pytest.raises(ValueError, match="keep_override"):   # sub-layer masks: [n_masks = 2][B]
        ld.ld_layer_fwd(sub, {k: 16 for k in ld.WEIGHT_KEYS}, 0, 0.1, 0, 0, 16, 16,
                        keep_override=torch.zeros(2, dtype=torch.uint8), stream=0)
    with pytest.raises(ValueError, match="layers"):
        ld.ld_stack_step(c, [w, w], [0.1], 0, 0, 16, 16, [dw], torch.zeros(8, dtype=torch.uint8))
