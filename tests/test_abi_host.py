"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host-only logic (the boundary rule, workspace sizing, argument
validation that returns before any launch) is right.  No device is touched:
device pointers passed here are dummies that validation never dereferences.
"""
import os
import re
import subprocess

import numpy as np
import pytest

from oracle.boundary import strict_prefix_boundary as brute_boundary
from paper_2609_15030_amd import linattn as la

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "linattn.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(la.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", la.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for n in names:
        assert n in exported, n
        assert hasattr(la.library(), n)


def test_library_targets_gfx950_only():
    """The offload bundle ids embedded in the built library name gfx950 only."""
    data = open(la.LIB_PATH, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa-+(gfx\w+)", data))
    assert targets == {b"gfx950"}


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


@pytest.mark.parametrize("row", _rows("table4_boundary_matrix.txt"), ids=lambda r: r[0])
def test_library_boundary_reproduces_table4(row):
    N, B_after, suffix = int(row[0]), int(row[4]), int(row[5])
    assert la.strict_prefix_boundary(N, 1792, N) == B_after
    assert N - B_after == suffix


def test_library_boundary_matches_brute_force():
    for C in list(range(1, 40)) + [64, 256, 1024, 1792]:
        for N in list(range(1, 300)) + [3583, 3584, 3585, 5375, 5376, 5377, 32768]:
            for avail in (0, 1, C - 1, C, 2 * C + 1, N - 1, N, N + C, 10 ** 6):
                if avail < 0:
                    continue
                assert la.strict_prefix_boundary(N, C, avail) == brute_boundary(N, C, avail), (N, C, avail)


def test_library_boundary_rejects_invalid():
    for args in [(0, 16, 0), (-5, 16, 3), (10, 0, 10), (10, -2, 10), (10, 4, -1)]:
        st, b = la.strict_prefix_boundary_status(*args)
        assert st == la.LA_ERR_INVALID_ARG and b == -1
    assert la.library().strict_prefix_boundary(10, 4, 10, None) == la.LA_ERR_INVALID_ARG


def test_workspace_bytes():
    sh = la.make_shape(1, 8, 128, 128, 256)
    a = la.la_prefill_workspace_bytes(sh, 3584)
    b = la.la_prefill_workspace_bytes(sh, 7168)
    assert 0 < a < b
    # 56 chunks x 8 heads x (X fragments 6 KB + gate block 1 KB)
    assert a >= 56 * 8 * 7 * 1024


FAKE = 1 << 20          # 16-byte aligned dummy device address (never dereferenced)


def _resume_status(shape, cu, starts, ws_bytes=1 << 40):
    lib = la.library()
    cu = np.asarray(cu, np.int32)
    starts = np.asarray(starts, np.int64)
    P = lambda a: a.ctypes.data_as(la.ctypes.c_void_p)
    return lib.la_prefill_resume(la.ctypes.byref(shape), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, P(cu),
                                 FAKE, P(starts), FAKE, FAKE, FAKE, None, None, None,
                                 FAKE, ws_bytes, None)


def test_resume_rejects_empty_suffix_before_launch():
    sh = la.make_shape(2, 8, 128, 128, 256)
    assert _resume_status(sh, [0, 256, 256], [3328, 3584]) == la.LA_ERR_EMPTY_SUFFIX
    assert "empty suffix" in la.last_error_message()


def test_resume_rejects_misaligned_state_before_launch():
    sh = la.make_shape(1, 8, 128, 128, 256)
    assert _resume_status(sh, [0, 256], [3327]) == la.LA_ERR_MISALIGNED_STATE


def test_resume_rejects_bad_tables_and_shapes():
    sh = la.make_shape(1, 8, 128, 128, 256)
    assert _resume_status(sh, [5, 256], [0]) == la.LA_ERR_INVALID_ARG          # cu[0] != 0
    assert _resume_status(la.make_shape(2, 8, 128, 128, 256), [0, 300, 200], [0, 0]) == la.LA_ERR_INVALID_ARG
    assert _resume_status(sh, [0, 256], [-256]) == la.LA_ERR_INVALID_ARG
    assert _resume_status(la.make_shape(1, 8, 96, 128, 256), [0, 256], [0]) == la.LA_ERR_UNSUPPORTED
    assert _resume_status(la.make_shape(1, 8, 128, 128, 256, chunk=32), [0, 256], [0]) == la.LA_ERR_UNSUPPORTED
    assert _resume_status(la.make_shape(1, 8, 128, 128, 256, io_dtype=7), [0, 256], [0]) == la.LA_ERR_INVALID_ARG
    assert _resume_status(la.make_shape(1, 8, 128, 128, 256, variant=3), [0, 256], [0]) == la.LA_ERR_INVALID_ARG
    assert _resume_status(la.make_shape(0, 8, 128, 128, 256), [0], []) == la.LA_ERR_INVALID_ARG


def test_short_workspace_is_rejected_before_launch():
    sh = la.make_shape(1, 8, 128, 128, 256)
    need = la.la_prefill_workspace_bytes(sh, 256)
    assert _resume_status(sh, [0, 256], [3328], ws_bytes=need - 1) == la.LA_ERR_WORKSPACE


def test_paged_validation_before_launch():
    lib = la.library()
    assert lib.la_state_save_paged(FAKE, 4, 6, FAKE, 8, FAKE, None, None) == la.LA_ERR_INVALID_ARG
    assert lib.la_state_restore_paged(FAKE, 8, FAKE, FAKE, 4, 0, None, None) == la.LA_ERR_INVALID_ARG
    assert lib.la_state_save_paged(FAKE + 4, 4, 8, FAKE, 8, FAKE, None, None) == la.LA_ERR_INVALID_ARG
    assert lib.la_state_save_paged(FAKE, 0, 8, FAKE, 8, FAKE, None, None) == la.LA_OK   # nothing to do


def test_resume_state_validation_before_launch():
    lib = la.library()
    sh = la.make_shape(1, 1, 64, 64, 16)
    cu = np.array([0, 64], np.int32)
    P = la.ctypes.c_void_p
    ws = lib.la_prefill_workspace_bytes(la.ctypes.byref(sh), 64)

    def call(state_in=None, starts=(16,)):
        st = np.asarray(starts, np.int64)
        return lib.la_prefill_resume(la.ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, P(cu.ctypes.data),
                                     P(cu.ctypes.data), FAKE, P(st.ctypes.data), state_in, FAKE, FAKE, None,
                                     None, None, FAKE, ws, None)
    assert call(state_in=None) == la.LA_ERR_INVALID_ARG                  # resume without a state
    assert call(state_in=FAKE, starts=[8]) == la.LA_ERR_MISALIGNED_STATE
    assert call(state_in=FAKE + 4) == la.LA_ERR_INVALID_ARG              # misaligned state


def test_prefill_form_is_a_function_of_the_shape():
    """The kernels a call runs depend on dtype, head dims and C only (never
    on lengths), so a resume runs the arithmetic of the run that wrote its
    checkpoint: bf16 takes the fused scan, or the two-level fused scan from
    C > 448 (8 chunks per interval); fp32 the one-tile scan with its output
    wave (dk = 64) or the dk-split scan (dk = 128)."""
    F = la.la_prefill_form
    for d in (64, 128):
        for C in (16, 64, 256, 448):
            assert F(la.make_shape(3, 8, d, 128, C, la.LA_BF16)) == la.LA_FORM_FUSED_SCAN
        for C in (449, 512, 1024, 1792):
            assert F(la.make_shape(3, 8, d, 128, C, la.LA_BF16)) == la.LA_FORM_FUSED_TWO_LEVEL
    assert F(la.make_shape(1, 1, 64, 64, 16, la.LA_F32)) == la.LA_FORM_TILE_SCAN_OUT
    assert F(la.make_shape(1, 1, 64, 128, 1024, la.LA_F32)) == la.LA_FORM_TILE_SCAN_OUT
    assert F(la.make_shape(1, 1, 128, 64, 16, la.LA_F32)) == la.LA_FORM_SPLIT_DK_SCAN
    assert F(la.make_shape(1, 1, 96, 128, 16)) == la.LA_FORM_NONE


def test_scan_columns_follow_the_chain_counts():
    """The fused scan's column widths are a scheduling choice made from the
    chains' chunk counts: 128 columns once the chains give every CU two
    workgroups; else the longest chains (a multiple of 8, or all) at 32
    columns and the rest at 64, as many narrow as shortens the estimated
    span: all of one sequence's chains, none of many even ones, the longest
    sequences of a batch whose longest chains dominate.  The call reports
    (width, narrow chains), with 64 for a mix.  fp32 runs no fused scan
    (0), nor does an invalid call."""
    W = la.la_prefill_scan_columns
    cu = lambda lens: np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    sh = lambda n, H=8, C=256, io=la.LA_BF16, d=128: la.make_shape(n, H, d, d, C, io)
    assert W(sh(1), cu([3584])) == (32, 8)                    # one TP rank's 8 chains
    assert W(sh(32), cu([3584] * 32)) == (64, 0)              # 256 even chains
    assert W(sh(64), cu([300] * 64)) == (128, 0)              # 512 chains
    # the strict-prefix suffixes of the 16-sequence varlen step, and the
    # same batch all cold: the two (four) longest sequences run narrow
    step = [8064, 7760, 6080, 5136, 4096, 4000, 3840, 3136, 1632, 1504, 960, 368, 240, 176, 176, 80]
    cold = [7760, 8016, 5376, 8064, 3136, 4000, 2656, 5136, 6080, 6320, 4096, 1216, 3696, 7152, 1968, 2784]
    assert W(sh(16), cu(step)) == (64, 16)
    assert W(sh(16), cu(cold)) == (64, 32)
    # the two-level form's replay: (sequence, head, segment) units
    assert W(sh(1, 16, 1024), cu([32768])) == (128, 0)        # 16 x 32 segments
    assert W(sh(1, 8, 1792), cu([3584])) == (64, 0)           # 8 x 2 segments
    rng = np.random.default_rng(9)
    for _ in range(50):                                        # narrow chains: none, all, or a multiple of 8
        n, H = int(rng.integers(1, 40)), int(rng.integers(1, 12))
        w, k = W(sh(n, H, 64), cu(rng.integers(0, 3000, n)))
        assert w in (32, 64, 128) and (k == n * H if w == 32 else (k % 8 == 0 and k < n * H))
        assert w != 128 or (k == 0 and n * H >= 512)
    assert W(sh(1, d=64), cu([3584])) == (64, 0)               # other head sizes: 64 only
    assert W(sh(1, io=la.LA_F32), cu([3584])) == (0, 0)
    assert W(la.make_shape(1, 1, 96, 128, 16), cu([10])) == (0, 0)
    assert W(sh(2), np.array([0, 10, 5], np.int32)) == (0, 0)  # decreasing offsets
    assert W(sh(1), np.array([3, 10], np.int32)) == (0, 0)     # offsets must start at 0


def test_checkpoint_rows_match_absolute_multiples():
    """la_checkpoint_rows numbers the multiples of C in (B_i, B_i + len_i]
    consecutively, sequence after sequence (brute force over positions)."""
    rng = np.random.default_rng(7)
    for _ in range(200):
        n = int(rng.integers(1, 9))
        C = int(rng.choice([1, 16, 64, 256, 1792]))
        lens = rng.integers(0, 5 * C + 3, n)
        starts = None if rng.random() < 0.3 else C * rng.integers(0, 6, n)
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        offs, total = la.la_checkpoint_rows(cu, starts, C)
        row = 0
        for i in range(n):
            b = 0 if starts is None else int(starts[i])
            assert offs[i] == row
            row += sum(1 for p in range(b + 1, b + int(lens[i]) + 1) if p % C == 0)
        assert total == row
    with pytest.raises(la.LinAttnError):
        la.la_checkpoint_rows(np.array([0, 5, 3], np.int32), None, 16)
    with pytest.raises(la.LinAttnError):
        la.la_checkpoint_rows(np.array([0, 5], np.int32), None, 0)


def test_workspace_holds_only_what_the_form_uses():
    """bf16 calls keep 7 KB per chunk slot and head (X fragments and the
    gate block), plus the segment regions of the two-level scan; fp32 calls
    keep the per-chunk operands, and the dk-split form also the per-chunk
    states and U its output kernel reads."""
    def ws(n_seqs, H, dk, dv, C, io, tokens):
        return la.la_prefill_workspace_bytes(la.make_shape(n_seqs, H, dk, dv, C, io), tokens)
    # varlen batch: 16 sequences, 77,456 tokens, 8 heads, C = 256 (1,217 chunk slots at most)
    slots = (77456 + 255 * 16) // 256 * 4
    got = ws(16, 8, 128, 128, 256, la.LA_BF16, 77456)
    assert got <= slots * 8 * (6 * 1024 + 1024) + 4096
    assert got < 0.1 * 1.15 * 2 ** 30            # the operand workspace of the unfused path was 1.15 GiB
    # two-level (C = 1024, 16 chunks per segment): + Phi' (bf16) + R + D + entering state per segment-head
    one = ws(1, 16, 128, 128, 1024, la.LA_BF16, 32768)
    segs = 32 * 16
    assert one >= 512 * 16 * 7 * 1024 + segs * (128 * 128 * 2 + 2 * 128 * 128 * 4)
    # fp32 forms: the split-dk scan needs the per-chunk states and U, the one-tile form does not
    a64 = ws(1, 1, 64, 64, 16, la.LA_F32, 256)
    a128 = ws(1, 1, 128, 64, 16, la.LA_F32, 256)
    slots32 = 16
    assert a128 - a64 >= slots32 * (128 * 64 * 4 + 64 * 64 * 4)


def test_paged_prefill_validation_before_launch():
    lib = la.library()
    sh = la.make_shape(1, 1, 64, 64, 16)
    cu = np.array([0, 64], np.int32)
    offs = np.array([0], np.int32)
    P = la.ctypes.c_void_p
    ws = lib.la_prefill_workspace_bytes(la.ctypes.byref(sh), 64)

    def call(pool=FAKE, ck=None, st_ids=None, starts=None, offsets=True, n_pages=4, null_pages=False):
        pg = la.LaPages(pool, n_pages, ck, st_ids, None)
        st = None if starts is None else np.asarray(starts, np.int64)
        return lib.la_prefill_paged(la.ctypes.byref(sh), None if null_pages else la.ctypes.byref(pg),
                                    FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, P(cu.ctypes.data),
                                    FAKE if st is not None else None, P(st.ctypes.data) if st is not None else None,
                                    FAKE, FAKE, FAKE if offsets else None, P(offs.ctypes.data) if offsets else None,
                                    FAKE, ws, None)
    assert call(null_pages=True) == la.LA_ERR_INVALID_ARG
    assert call(st_ids=FAKE) == la.LA_ERR_INVALID_ARG                     # starting pages, cold call
    assert call(starts=[16]) == la.LA_ERR_INVALID_ARG                      # resume without starting pages
    assert call(pool=None, ck=FAKE) == la.LA_ERR_INVALID_ARG               # page ids without a pool
    assert call(pool=FAKE + 4, ck=FAKE) == la.LA_ERR_INVALID_ARG           # misaligned pool
    assert call(ck=FAKE, offsets=False) == la.LA_ERR_INVALID_ARG           # checkpoint pages need row offsets
    assert call(ck=FAKE, n_pages=-1) == la.LA_ERR_INVALID_ARG
    assert call(ck=FAKE, n_pages=1 << 31) == la.LA_ERR_INVALID_ARG
    assert call(st_ids=FAKE, starts=[8]) == la.LA_ERR_MISALIGNED_STATE


@pytest.mark.parametrize("seed", range(3))
def test_library_hybrid_boundary_matches_oracle(seed):
    from oracle.boundary import hybrid_boundary
    rng = np.random.default_rng(100 + seed)
    for _ in range(400):
        bt = int(rng.choice([1, 4, 16, 64]))
        C = bt * int(rng.integers(1, 8))
        N = int(rng.integers(1, 10 * C))
        kv, stc = int(rng.integers(0, 10 * C)), int(rng.integers(0, 10 * C))
        assert la.la_hybrid_boundary(N, C, bt, kv, stc) == hybrid_boundary(N, C, bt, kv, stc)
    for bad in [(0, 16, 16, 0, 0), (10, 0, 16, 10, 10), (10, 16, 0, 10, 10), (10, 16, 16, -1, 10)]:
        with pytest.raises(la.LinAttnError) as e:
            la.la_hybrid_boundary(*bad)
        assert e.value.status == la.LA_ERR_INVALID_ARG
    with pytest.raises(la.LinAttnError) as e:
        la.la_hybrid_boundary(5376, 1792, 48, 5376, 5376)
    assert e.value.status == la.LA_ERR_MISALIGNED_STATE


def test_hybrid_restore_validation_before_launch():
    lib = la.library()
    P = la.ctypes.c_void_p

    def call(bounds, block_tokens=16, block_bytes=1024, max_blocks=8, kv_null=False, n_heads=2, bdev=True):
        kv = la.LaKvBlocks(FAKE, 64, FAKE, 64, block_bytes, block_tokens, FAKE, FAKE, max_blocks)
        b = np.asarray(bounds, np.int64)
        return lib.la_hybrid_restore(None if kv_null else la.ctypes.byref(kv), len(b), n_heads, 16,
                                     FAKE if bdev else None, P(b.ctypes.data) if len(b) else None, FAKE, 4,
                                     FAKE, FAKE, None, None)
    assert call([16], kv_null=True) == la.LA_ERR_INVALID_ARG
    assert call([]) == la.LA_OK                                          # nothing to restore
    assert call([24]) == la.LA_ERR_MISALIGNED_STATE                      # not a whole number of blocks
    assert call([16 * 9]) == la.LA_ERR_INVALID_ARG                       # more blocks than max_blocks
    assert call([16], block_bytes=1000) == la.LA_ERR_INVALID_ARG         # not a multiple of 16
    assert call([16], block_tokens=0) == la.LA_ERR_INVALID_ARG
    assert call([-16]) == la.LA_ERR_INVALID_ARG
    assert call([16], bdev=False) == la.LA_ERR_INVALID_ARG


def test_decode_validation_before_launch():
    lib = la.library()
    sh = la.make_shape(2, 8, 128, 128, 256)
    ok = [FAKE] * 7
    for i in range(7):                      # every buffer is required
        args = list(ok)
        args[i] = None
        assert lib.la_decode_step(la.ctypes.byref(sh), *args, None) == la.LA_ERR_INVALID_ARG
    # state misaligned; q misaligned for bf16
    assert lib.la_decode_step(la.ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 4, FAKE,
                              None) == la.LA_ERR_INVALID_ARG
    assert lib.la_decode_step(la.ctypes.byref(sh), FAKE + 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                              None) == la.LA_ERR_INVALID_ARG
    bad = la.make_shape(2, 8, 96, 128, 256)
    assert lib.la_decode_step(la.ctypes.byref(bad), *ok, None) == la.LA_ERR_UNSUPPORTED
    assert lib.la_decode_step(None, *ok, None) == la.LA_ERR_INVALID_ARG


def test_status_strings():
    assert la.status_string(la.LA_ERR_EMPTY_SUFFIX) == "LA_ERR_EMPTY_SUFFIX"
    assert la.status_string(99) == "LA_ERR_UNKNOWN"
