"""tt_verify_noalloc (the library's own scratch, no workspace) against tt_verify on the same
inputs, called through the C-ABI twice in a row, the second call with a smaller batch: both
the split path (few streams, chunk sums in the scratch) and the one-workgroup-per-stream path
with residual rows (Z and the selected row in the scratch)."""
import numpy as np
import pytest

from gpu_util import oracle_run, to_dev, upload
from paper_2510_15545_amd import synth

pytestmark = pytest.mark.gpu


def _verify_both(wl, residual):
    import torch

    import paper_2510_15545_amd as tt

    d = upload(wl)
    q = to_dev(oracle_run(wl)["q"])
    args = (wl.v_t, d["verify_ids"], d["target_off"], q, d["target_probs"], d["u_accept"], d["u_sample"],
            max(0, wl.max_m))
    ref = tt.verify(*args, residual=residual)
    got = tt.verify_noalloc(*args, residual=residual)
    torch.cuda.synchronize()
    assert np.array_equal(got[0].cpu().numpy(), ref[0].cpu().numpy())
    assert np.array_equal(got[1].cpu().numpy(), ref[1].cpu().numpy())
    if residual:
        assert np.array_equal(got[2].cpu().numpy().view(np.uint32), ref[2].cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("c,n_big,n_small,residual", [(2, 32, 5, True), (1, 300, 260, True), (3, 256, 40, False)])
def test_noalloc_matches_verify_twice(c, n_big, n_small, residual):
    print(f"[case] tt_verify_noalloc workload {c} streams {n_big} then {n_small}", flush=True)
    _verify_both(synth.make(c, n_streams=n_big), residual)
    _verify_both(synth.make(c, n_streams=n_small, seed_shift=1), residual)


def test_noalloc_refuses_batches_past_its_scratch():
    import ctypes

    import paper_2510_15545_amd as tt

    n = ctypes.c_size_t(0)
    assert tt.lib().tt_verify_workspace_size(8192, 151936, ctypes.byref(n)) == 0 and n.value > 8 << 20
    dummy = ctypes.c_void_p(256)
    st = tt.lib().tt_verify_noalloc(8192, 151936, dummy, dummy, dummy, dummy, 151936, dummy, dummy, 8, dummy, dummy,
                                    None, None)
    assert st == tt.TT_EWORKSPACE
