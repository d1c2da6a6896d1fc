"""Run a synth.Workload through the GPU library and through the oracle; compare."""
import numpy as np

import oracle
import paper_2510_15545_amd as tt


def to_dev(a, dtype=None):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def upload(wl):
    """Device copies of a workload's arrays (dict of torch tensors)."""
    import torch

    d = {
        "vd": tt.Vocab.from_host(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_d.max_len),
        "vt": tt.Vocab.from_host(wl.vocab_t.data, wl.vocab_t.offsets, wl.vocab_t.max_len),
        "draft_ids": to_dev(wl.draft_ids), "draft_off": to_dev(wl.draft_off),
        "target_ids": to_dev(wl.target_ids), "target_off": to_dev(wl.target_off),
    }
    if wl.draft_probs is not None:
        d["draft_probs"] = to_dev(wl.draft_probs)
        d["target_probs"] = to_dev(wl.target_probs)
        d["verify_ids"] = to_dev(wl.verify_ids)
        d["u_accept"] = to_dev(wl.u_accept)
        d["u_sample"] = to_dev(wl.u_sample)
    torch.cuda.synchronize()
    return d


def gpu_align(wl, d, w=None, bounds=None):
    """tt_align over the workload; `bounds` = (max_k, max_m) passed instead of the batch's own
    maxima (larger bounds move short pairs from the row-scan kernel to the strip kernel)."""
    w = wl.w if w is None else w
    mk, mm = (max(1, wl.max_k), max(1, wl.max_m)) if bounds is None else bounds
    return tt.align(d["vd"], d["vt"], d["draft_ids"], d["draft_off"], d["target_ids"], d["target_off"],
                    w, mk, mm, n_path=tt.path_capacity(wl.draft_off[-1], wl.target_off[-1]))


def gpu_run(wl, w=None, residual=False, d=None, bounds=None):
    """align -> transfer -> verify on the GPU; returns host numpy arrays."""
    import torch

    d = upload(wl) if d is None else d
    cost, plen, path, mp = gpu_align(wl, d, w, bounds)
    out = {"cost": cost, "path_len": plen, "path": path, "map": mp}
    if wl.draft_probs is not None:
        q = tt.transfer(wl.v_d, d["draft_ids"], d["draft_off"], d["target_off"], mp, d["draft_probs"])
        nacc, tok, res = tt.verify(wl.v_t, d["verify_ids"], d["target_off"], q, d["target_probs"],
                                   d["u_accept"], d["u_sample"], max(0, wl.max_m), residual=residual)
        out.update(q=q, n_accepted=nacc, out_token=tok, residual=res)
    torch.cuda.synchronize()
    m_total = int(wl.target_off[-1])
    host = {}
    for k, v in out.items():
        if v is None:
            host[k] = None
            continue
        a = v.cpu().numpy()
        if k in ("map", "q"):
            a = a[:m_total]
        host[k] = a
    return host


def compare_align(wl, g, o):
    assert np.array_equal(g["cost"], o["cost"]), np.nonzero(g["cost"] != o["cost"])
    assert np.array_equal(g["path_len"], o["path_len"])
    assert np.array_equal(g["map"], o["map"])
    for b in range(wl.n):
        base = 2 * (int(wl.draft_off[b]) + int(wl.target_off[b]))
        n = 2 * int(o["path_len"][b])
        assert np.array_equal(g["path"][base:base + n], o["path"][base:base + n]), b


def compare_verify(g, o, residual=False):
    qg, qo = g["q"], o["q"]
    assert np.array_equal(qg.view(np.uint32), qo.view(np.uint32)) or \
        np.array_equal(np.isnan(qg), np.isnan(qo)) and np.array_equal(qg[~np.isnan(qg)], qo[~np.isnan(qo)])
    assert np.array_equal(g["n_accepted"], o["n_accepted"]), np.nonzero(g["n_accepted"] != o["n_accepted"])
    assert np.array_equal(g["out_token"], o["out_token"]), np.nonzero(g["out_token"] != o["out_token"])
    if residual:
        rg, ro = g["residual"], o["residual"]
        ro = ro[:, :rg.shape[1]] if ro.shape[1] >= rg.shape[1] else ro
        rg = rg[:, :ro.shape[1]]
        diff = np.abs(rg.astype(np.float64) - ro.astype(np.float64))
        tol = 1e-6 * np.abs(ro.astype(np.float64))
        assert np.all(diff <= tol), float((diff - tol).max())


def oracle_run(wl, w=None, residual=False, n_threads=None):
    if w is not None and w != wl.w:
        import copy

        wl = copy.copy(wl)
        wl.w = w
    return oracle.run_workload(wl, n_threads=n_threads, residual=residual)
