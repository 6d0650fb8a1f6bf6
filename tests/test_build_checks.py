"""CPU tests of the assembly checks that build.py applies to every device
object: the untracked-activation-load hazard scan and the MFMA operand
overlap scan, on small hand-written assembly listings."""
from paper_2504_15299_amd import build

HEAD = "_Zkernel:\n"

SAFE = HEAD + """
\ts_and_saveexec_b64 s[4:5], s[6:7]
\tglobal_load_dwordx4 v[0:3], v[16:17], off
\ts_mov_b64 exec, s[4:5]
\tglobal_load_lds_dwordx4 v[40:41], off
\tglobal_load_lds_dwordx4 v[42:43], off
\ts_cbranch_vccnz .LBB0_2
\tv_mov_b32_e32 v20, v21
\tglobal_load_lds_dwordx4 v[44:45], off
.LBB0_2:
\ts_waitcnt vmcnt(2)
\tv_mfma_scale_f32_16x16x128_f8f6f4 v[24:27], v[32:35], v[0:7], 0, v8, v9 op_sel_hi:[0,0,0] cbsz:4
\tv_mov_b32_e32 v0, 0
\ts_endpgm
"""

# the same listing with a copy through the load's registers on one branch
# only, before the covering wait: the data can land after the copy
HAZARD = SAFE.replace("\tv_mov_b32_e32 v20, v21\n", "\tv_readfirstlane_b32 s44, v1\n")

# a compiler-tracked load whose address overlaps the pending one
TRACKED_OVERLAP = SAFE.replace("\tv_mov_b32_e32 v20, v21\n",
                               "\tglobal_load_dwordx4 v[20:23], v[2:3], off\n")
# a later load into the same registers is fine: loads complete in order
TRACKED_WAW = SAFE.replace("\tv_mov_b32_e32 v20, v21\n",
                           "\tglobal_load_dwordx4 v[0:3], v[20:21], off\n")

# a use after vmcnt(0) on every path is fine
AFTER_DRAIN = HEAD + """
\ts_and_saveexec_b64 s[4:5], s[6:7]
\tglobal_load_dwordx4 v[0:3], v[16:17], off
\ts_mov_b64 exec, s[4:5]
\ts_waitcnt vmcnt(0)
\tv_mov_b32_e32 v5, v0
\ts_endpgm
"""


def test_untracked_load_check_accepts_safe_listing():
    assert build.untracked_load_hazards(SAFE) == []
    assert build.untracked_load_hazards(AFTER_DRAIN) == []
    # a copy after a covering wait (two DMA instructions issued after the
    # load on either path, vmcnt(2)) is fine
    covered = SAFE.replace("\tv_mov_b32_e32 v0, 0\n", "\tv_mov_b32_e32 v50, v1\n")
    assert build.untracked_load_hazards(covered) == []


def test_untracked_load_check_finds_use_on_a_branch():
    bad = build.untracked_load_hazards(HAZARD)
    assert len(bad) == 1
    assert "readfirstlane" in bad[0][2]


def test_untracked_load_check_sees_overlapping_tracked_loads():
    bad = build.untracked_load_hazards(TRACKED_OVERLAP)
    assert len(bad) == 1
    assert "v[2:3]" in bad[0][2]
    assert build.untracked_load_hazards(TRACKED_WAW) == []


# an inline-asm load (no EXEC narrowing), as the 4-wave GEMM kernels issue
# their activation operands: the copy before the covering wait is flagged,
# the same copy after vmcnt(1) (one DMA issued after the load) is not
ASM_LOAD = HEAD + """
	;;#ASMSTART
	global_load_dwordx4 v[8:11], v[2:3], off
	;;#ASMEND
	global_load_lds_dwordx4 v[40:41], off
	COPY_BEFORE
	s_waitcnt vmcnt(1)
	v_mov_b32_e32 v20, v9
	s_endpgm
"""


def test_untracked_load_check_covers_inline_asm_loads():
    assert build.untracked_load_hazards(ASM_LOAD.replace("\tCOPY_BEFORE\n", "")) == []
    bad = build.untracked_load_hazards(ASM_LOAD.replace("COPY_BEFORE", "v_mov_b32_e32 v21, v10"))
    assert len(bad) == 1 and "v10" in bad[0][2]


def test_mfma_overlap_check():
    ok = "\tv_mfma_f32_16x16x32_bf16 v[0:3], v[4:7], v[8:11], v[0:3]\n"
    bad = "\tv_mfma_f32_16x16x32_bf16 v[4:7], v[4:7], v[8:11], 0\n"
    assert build.mfma_overlaps(ok) == []
    assert len(build.mfma_overlaps(bad)) == 1


# a 64-bit scalar address add split around an inline-asm block that writes
# SCC: the carry the second half reads is the asm's, not the first half's
SCC_LIVE = HEAD + """
\ts_add_u32 s30, s30, s62
\t;;#ASMSTART
\ts_and_saveexec_b64 s[38:39], s[4:5]
\tglobal_load_dwordx4 v[0:3], v[10:11], off
\ts_mov_b64 exec, s[38:39]
\t;;#ASMEND
\ts_addc_u32 s31, s31, s36
\ts_endpgm
"""

# the same asm with the add completed before it
SCC_DEAD = HEAD + """
\ts_add_u32 s30, s30, s62
\ts_addc_u32 s31, s31, s36
\t;;#ASMSTART
\ts_and_saveexec_b64 s[38:39], s[4:5]
\tglobal_load_dwordx4 v[0:3], v[10:11], off
\ts_mov_b64 exec, s[38:39]
\t;;#ASMEND
\ts_cmp_eq_u32 s2, 0
\ts_cbranch_scc1 .LBB0_1
.LBB0_1:
\ts_endpgm
"""


def test_scc_check_finds_carry_across_asm():
    bad = build.scc_clobber_hazards(SCC_LIVE)
    assert len(bad) == 1 and bad[0][1].startswith("s_addc_u32")
    assert build.scc_clobber_hazards(SCC_DEAD) == []


def test_kernel_source_hash_ignores_comments(tmp_path, monkeypatch):
    """The hash that gates the committed HBM byte counters changes with the
    decode kernels' code, not with their comments or blank space."""
    import bench
    src = tmp_path / "paper_2504_15299_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "internal.h").write_text("int f(int x) { return x; }\n")
    (src / "ffn_decode.hip").write_text("// a kernel\nint g(int y) {\n  return y + 1;  // add one\n}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash()
    (src / "ffn_decode.hip").write_text("/* the kernel */\nint g(int y)   {\n\n  return y + 1;\n}\n")
    assert bench.kernel_source_hash() == h0
    (src / "ffn_decode.hip").write_text("int g(int y) { return y + 2; }\n")
    assert bench.kernel_source_hash() != h0


LDS_OK = HEAD + """
\t;;#ASMSTART
\tds_read_b32 v10, v40 offset:256
\t;;#ASMEND
\t;;#ASMSTART
\tds_read_b64 v[12:13], v41 offset:512
\t;;#ASMEND
\tv_mov_b32_e32 v20, v21
\t;;#ASMSTART
\ts_waitcnt lgkmcnt(0)
\t;;#ASMEND
\tv_add_u32_e32 v22, v10, v12
\ts_endpgm
"""
# the compiler reuses the pending read's register for another value
LDS_BAD = LDS_OK.replace("\tv_mov_b32_e32 v20, v21\n", "\tv_mov_b32_e32 v10, v21\n")
# a later batched read addresses through the pending register
LDS_BAD_ADDR = LDS_OK.replace("ds_read_b64 v[12:13], v41", "ds_read_b64 v[12:13], v10")


def test_asm_lds_read_check():
    assert build.asm_lds_read_hazards(LDS_OK) == []
    assert len(build.asm_lds_read_hazards(LDS_BAD)) == 1
    assert len(build.asm_lds_read_hazards(LDS_BAD_ADDR)) == 1
