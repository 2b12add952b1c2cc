"""Helpers for GPU tests: run the HIP library on a numpy mask, compare to the oracle."""
import sys

import numpy as np

from invariants import check_index_valid

RTOL, ATOL = 1e-5, 1e-6     # float tolerance for sampled distances


def announce(msg):
    """Name the case before a GPU step, so a fault report says what ran."""
    print("[gpu case] " + msg, flush=True)
    sys.stdout.flush()


def run_gpu(mask, ndim, sampling=None, dist=True, idx=False, sq=False, stream=None):
    """mask: numpy (batch..., *spatial) uint8. Returns dict of numpy results."""
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    x = torch.from_numpy(np.ascontiguousarray(mask)).to(dev)
    lead = mask.shape[:mask.ndim - ndim]
    spatial = mask.shape[mask.ndim - ndim:]
    out = {}
    d = torch.empty(mask.shape, dtype=torch.float32, device=dev) if dist else None
    i = torch.empty(lead + (ndim,) + spatial, dtype=torch.int32, device=dev) if idx else None
    if dist or idx:
        binding.tm_edt(x, ndim, sampling, d, i, stream=stream)
    s = None
    if sq:
        s = torch.empty(mask.shape, dtype=torch.int32, device=dev)
        binding.tm_edt_sq(x, ndim, s, None, stream=stream)
    torch.cuda.synchronize()
    out["dist"] = None if d is None else d.cpu().numpy()
    out["idx"] = None if i is None else i.cpu().numpy()
    out["sq"] = None if s is None else s.cpu().numpy()
    return out


def assert_close(got, want, what):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    err = np.abs(got - want)
    ok = (err <= RTOL * np.abs(want)) | (err <= ATOL)
    if not ok.all():
        k = np.argwhere(~ok)[0]
        raise AssertionError("%s: %d of %d elements outside 1e-5 rel / 1e-6 abs; first at %s: "
                             "got %r want %r" % (what, int((~ok).sum()), ok.size, tuple(k),
                                                 got[tuple(k)], want[tuple(k)]))


def check_against_oracle(mask, ndim, sampling, res, ora):
    """Element-by-element comparison of one GPU result with the oracle's."""
    unit = sampling is None or all(float(s) == 1.0 for s in np.atleast_1d(sampling))
    if res.get("sq") is not None:
        assert np.array_equal(res["sq"], ora["sq"]), "int32 squared distances differ"
    if res.get("dist") is not None:
        if unit:
            # both sides are the correctly rounded sqrt of the same exact integer
            assert np.array_equal(res["dist"], ora["dist"]), "unit-sampling distances differ"
        else:
            assert_close(res["dist"], ora["dist"], "sampled distances")
    if res.get("idx") is not None:
        idx = res["idx"]
        lead = mask.shape[:mask.ndim - ndim]
        flat_mask = mask.reshape((-1,) + mask.shape[mask.ndim - ndim:])
        flat_idx = idx.reshape((-1, ndim) + mask.shape[mask.ndim - ndim:])
        if unit:
            # canonical: the nearest background element with the smallest flat index
            assert np.array_equal(idx, ora["idx"]), "indices differ from the canonical ones"
        else:
            sqd = ora["sqd"].reshape((-1,) + mask.shape[mask.ndim - ndim:])
            for b in range(flat_mask.shape[0]):
                bad = check_index_valid(flat_mask[b], sqd[b], flat_idx[b], sampling,
                                        rtol=2 * RTOL, atol=ATOL)
                assert bad == 0, "sample %d: %d indices are not nearest background" % (b, bad)
        del lead
