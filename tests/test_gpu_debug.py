"""The binding's debug mode on the GPU: with the check on, a batch whose device
copies equal the host copies runs and gives the same output as without the
check; a device copy that differs is refused before any launch."""
import pytest
import torch

from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W

pytestmark = pytest.mark.gpu


def test_debug_check_of_device_copies(monkeypatch):
    print("debug check tiny_single", flush=True)
    w = W.tiny_single()
    db = B.materialize(w, keep_host=[])
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    ref = cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale)
    monkeypatch.setattr(cw, "DEBUG_CHECK_COPIES", True)
    out = cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    db.meta.plan[12] += 1   # the header's work word: unused by the kernels, so harmless if launched
    sentinel = torch.full_like(out, 7.0)
    with pytest.raises(ValueError, match="plan"):
        cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale, out=sentinel)
    with pytest.raises(ValueError, match="plan"):
        cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    torch.cuda.synchronize()
    assert torch.all(sentinel == 7.0)
