"""Host-side validation of the attention-core calls: every case has exactly
one defect, so no call reaches a kernel; fake device addresses, skipped
wherever a GPU is visible."""
import pytest

from paper_2301_06813_amd import sbp

BF, F32 = sbp.SBP_BF16, sbp.SBP_F32
QA, KA, SA = 0x10000000, 0x20000000, 0x30000000


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


pytestmark = pytest.mark.skipif(_gpu_visible(), reason="uses fake device addresses")


def v4(ptr, B, H, R, C, dtype=BF, scope=sbp.SBP_GLOBAL, sb=None, sh=None, ld=None):
    ld = C if ld is None else ld
    sh = R * ld if sh is None else sh
    sb = H * sh if sb is None else sb
    return sbp.sbp_view4_t(ptr, B, H, R, C, sb, sh, ld, dtype, scope)


def _scores(**kw):
    # B 2, H 5 split over p 2: rank 1 holds 2 heads; Sq 64, Sk 48, D 32
    c = dict(q=v4(QA, 2, 5, 64, 32), k=v4(KA, 2, 5, 48, 32),
             s=v4(SA, 2, 2, 64, 48, F32, sbp.SBP_LOCAL), p=2, r=1)
    c.update(kw)
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_attn_scores(c["q"], c["k"], c["s"], c["p"], c["r"], stream=0)
    return ei.value.code


CASES = [
    ("rank out of range", dict(r=2), sbp.SBP_ERR_LAYOUT),
    ("no devices", dict(p=0), sbp.SBP_ERR_LAYOUT),
    ("fp32 input", dict(q=v4(QA, 2, 5, 64, 32, F32)), sbp.SBP_ERR_DTYPE),
    ("head dims differ", dict(k=v4(KA, 2, 5, 48, 40)), sbp.SBP_ERR_SHAPE),
    ("batches differ", dict(k=v4(KA, 3, 5, 48, 32)), sbp.SBP_ERR_SHAPE),
    ("global head counts differ", dict(k=v4(KA, 2, 6, 48, 32)), sbp.SBP_ERR_SHAPE),
    ("local head count is not rank 1's", dict(k=v4(KA, 2, 3, 48, 32, scope=sbp.SBP_LOCAL)),
     sbp.SBP_ERR_SHAPE),
    ("output heads", dict(s=v4(SA, 2, 3, 64, 48, F32, sbp.SBP_LOCAL)), sbp.SBP_ERR_SHAPE),
    ("output rows", dict(s=v4(SA, 2, 2, 48, 48, F32, sbp.SBP_LOCAL)), sbp.SBP_ERR_SHAPE),
    ("output heads overlap", dict(s=v4(SA, 2, 2, 64, 48, F32, sbp.SBP_LOCAL, sh=48)),
     sbp.SBP_ERR_SHAPE),
    ("ld < cols", dict(q=v4(QA, 2, 5, 64, 32, ld=16)), sbp.SBP_ERR_SHAPE),
    ("accumulate into bf16", dict(s=v4(SA, 2, 2, 64, 48, BF, sbp.SBP_ACCUMULATE)),
     sbp.SBP_ERR_DTYPE),
    ("misaligned", dict(q=v4(QA + 1, 2, 5, 64, 32)), sbp.SBP_ERR_ALIGN),
    ("output overlaps Q", dict(s=v4(QA + 4096, 2, 2, 64, 48, F32, sbp.SBP_LOCAL)),
     sbp.SBP_ERR_ALIAS),
    ("null data", dict(q=v4(None, 2, 5, 64, 32)), sbp.SBP_ERR_NULL),
]


@pytest.mark.parametrize("name,change,code", CASES, ids=[c[0] for c in CASES])
def test_scores_validation(name, change, code):
    assert _scores(**change) == code


def test_backward_validation():
    dS = v4(SA, 2, 5, 64, 48)
    q, k = v4(QA, 2, 5, 64, 32), v4(KA, 2, 5, 48, 32)
    dQ = v4(0x40000000, 2, 2, 64, 32, F32, sbp.SBP_LOCAL)
    dK = v4(0x40000000 + 4096, 2, 2, 48, 32, F32, sbp.SBP_LOCAL)   # overlaps dQ
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_attn_scores_bwd(dS, q, k, dQ, dK, 2, 1, stream=0)
    assert ei.value.code == sbp.SBP_ERR_ALIAS
    with pytest.raises(sbp.SbpError) as ei:   # dS columns must be the key length
        sbp.sbp_attn_scores_bwd(v4(SA, 2, 5, 64, 40), q, k,
                                v4(0x40000000, 2, 2, 64, 32, F32, sbp.SBP_LOCAL),
                                v4(0x50000000, 2, 2, 48, 32, F32, sbp.SBP_LOCAL), 2, 1, stream=0)
    assert ei.value.code == sbp.SBP_ERR_SHAPE
