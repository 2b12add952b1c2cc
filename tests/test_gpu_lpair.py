"""GPU parity of the packed whole-line pass (k_line_pair16: 16 adjacent
lines of up to 512 rows per workgroup, two lines per packed 16-bit word),
which unit-sampled distance passes take when their lines are a multiple of
16 rows long, 16 neighbouring lines are adjacent in memory, and there are at
least 512 groups of 16 lines.  Squared distances and distances must equal
the oracle's bit for bit.  The cases cover dense and sparse masks,
workgroups whose lines hold at most 32 site rows (the direct minimum),
distances of 256 and more with many site rows (the exact 32-bit re-search),
samples without background (the virtual element), the intermediate pass of a
3-D input, and squared-distance outputs."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu


def run_named(mask, nd):
    from paper_2608_24738_amd import binding
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, nd, None, dist=True, idx=False, sq=True)
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    return res, names


# kernel names: the row scan packs its distances to 16 bits (".o16") when the
# column pass is this one and every wave's rows pair up inside one block of
# rows; the first column pass then reads them (".i16")
PACKED = ("scan_word.o16", "line_pair_final.i16")


def check(mask, nd, tag, expect=PACKED):
    announce("line pair %s shape=%s" % (tag, mask.shape))
    res, names = run_named(mask, nd)
    for e in expect:
        assert e in names, names
    check_against_oracle(mask, nd, None, res, edt_oracle.edt(mask, nd, None, nthreads=16))


@pytest.mark.parametrize("p_bg", [0.3, 0.01, 0.0005, 0.00002])
def test_densities(p_bg):
    rng = np.random.default_rng([31, int(p_bg * 1e5)])
    mask = (rng.random((16, 512, 512)) >= p_bg).astype(np.uint8)
    check(mask, 2, "p_bg=%g" % p_bg)


def test_line_lengths():
    # 256-row columns (1024 wide, 8192 lines) and 64-row columns
    rng = np.random.default_rng(32)
    check((rng.random((8, 256, 1024)) >= 0.002).astype(np.uint8), 2, "n=256")     # 32-position words
    check((rng.random((16, 64, 8192)) >= 0.01).astype(np.uint8), 2, "n=64", expect=("line_pair_final",))


def test_packed_field_row_blocks():
    # rows of 64: a wave scans 32 rows of two 32-position words; blocks of 96
    # rows hold whole waves (packed field), blocks of 80 do not (int32 field)
    rng = np.random.default_rng(35)
    check((rng.random((128, 96, 64)) >= 0.05).astype(np.uint8), 2, "96x64 blocks")
    check((rng.random((128, 80, 64)) >= 0.05).astype(np.uint8), 2, "80x64 blocks",
          expect=("scan_word", "line_pair_final"))


def test_long_distances_many_sites():
    # every column's sites sit in rows 0..40 (41 site rows per workgroup, so
    # the search runs), and rows far below are 256 and more away: results of
    # 0xfffe and more are searched again on the exact copy
    mask = np.ones((16, 512, 512), np.uint8)
    mask[:, :41, 0] = 0
    mask[3, :41, 0] = 1
    mask[3, 500, 511] = 0          # one site row only: the direct minimum
    check(mask, 2, "long distances")


def test_samples_without_background():
    rng = np.random.default_rng(33)
    mask = (rng.random((16, 512, 512)) >= 0.001).astype(np.uint8)
    mask[0] = 1
    mask[7] = 1
    mask[8] = 0
    check(mask, 2, "empty samples")


def test_3d_intermediate_and_final():
    # workload 13 (2 x 256^3 balls): the axis-1 and axis-0 passes both take it
    mask = workloads.make_mask(13)[:, 0]
    check(mask, 3, "2x256^3 balls", expect=("scan_word.o16", "line_pair.i16", "line_pair_final"))


def test_full_workload_2():
    mask = workloads.make_mask(2)[:, 0]
    check(mask, 2, "32x512^2 discs")


def test_corner_blob():
    # background only in a 40 x 40 corner block: 40 site rows in every
    # workgroup (the search runs) and distances up to ~670 (most patches are
    # redone on the exact copy)
    mask = np.ones((16, 512, 512), np.uint8)
    mask[:, :40, :40] = 0
    mask[5, :40, :40] = 1
    mask[5, 300:340, 470:510] = 0
    check(mask, 2, "corner blob")
