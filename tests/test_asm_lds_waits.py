"""No kernel touches the registers of an inline-asm LDS read before its wait.

The check itself (asm_lds_check) is pinned first on small hand-written
assembly whose hazards are known, then run over the device assembly that the
library's own Makefile flags produce for the GEMM and attention kernels.
"""
import os
import shutil
import subprocess

import pytest

import asm_lds_check as chk

CSRC = os.path.join(os.path.dirname(__file__), "..", "paper_2609_13645_amd", "csrc")


def _kernel(body):
    """A one-kernel .s text; `asm:` marks an instruction written as inline asm."""
    out = ["_Z1kv:"]
    for line in body.strip().split("\n"):
        line = line.strip()
        if line.startswith("asm:"):
            out += [";;#ASMSTART", "\t" + line[4:].strip(), ";;#ASMEND"]
        else:
            out.append(line if line.endswith(":") else "\t" + line)
    out.append(".Lfunc_end0:")
    return "\n".join(out) + "\n"


def _hazards(tmp_path, body):
    p = tmp_path / "k.s"
    p.write_text(_kernel(body))
    res, n = chk.check_asm(str(p))
    return res["_Z1kv"], n


def test_use_before_wait_is_found(tmp_path):
    h, n = _hazards(tmp_path, """
        asm: ds_read_b64_tr_b16 v[10:11], v2
        v_bfi_b32 v20, s4, v10, v10
        s_waitcnt lgkmcnt(0)
        s_endpgm""")
    assert n == 1 and [x[1:] for x in h] == [("reads", [10], "v_bfi_b32 v20, s4, v10, v10")]


def test_use_after_covering_wait_is_clean(tmp_path):
    # two reads, lgkmcnt(1) retires the older one only
    h, _ = _hazards(tmp_path, """
        asm: ds_read_b128 v[10:13], v2
        asm: ds_read_b128 v[14:17], v3
        s_waitcnt lgkmcnt(1)
        v_mov_b32 v20, v13
        v_mov_b32 v21, v14
        s_waitcnt lgkmcnt(0)
        v_mov_b32 v22, v17
        s_endpgm""")
    assert [(x[1], x[2]) for x in h] == [("reads", [14])]


def test_compiler_lds_ops_count_towards_the_wait(tmp_path):
    # a compiler ds_write issued after the asm read is the newest LDS op, so
    # lgkmcnt(1) retires the asm read; a compiler read before it keeps it
    h, _ = _hazards(tmp_path, """
        asm: ds_read_b128 v[10:13], v2
        ds_write_b128 v5, v[30:33]
        s_waitcnt lgkmcnt(1)
        v_mov_b32 v20, v10
        ds_read_b128 v[40:43], v6
        asm: ds_read_b128 v[14:17], v3
        ds_bpermute_b32 v44, v7, v8
        s_waitcnt lgkmcnt(2)
        v_mov_b32 v21, v14
        s_waitcnt lgkmcnt(0)
        s_endpgm""")
    assert [(x[1], x[2]) for x in h] == [("reads", [14])]


def test_scalar_loads_do_not_retire_lds_reads(tmp_path):
    # SMEM may return first: lgkmcnt(1) with an s_load in flight does not
    # prove the asm read done
    h, _ = _hazards(tmp_path, """
        asm: ds_read_b128 v[10:13], v2
        s_load_dwordx2 s[0:1], s[4:5], 0x0
        s_waitcnt lgkmcnt(1)
        v_mov_b32 v20, v11
        s_endpgm""")
    assert [(x[1], x[2]) for x in h] == [("reads", [11])]


def test_overwrite_and_store_of_pending_registers(tmp_path):
    h, _ = _hazards(tmp_path, """
        asm: ds_read_b64_tr_b16 v[10:11], v2
        v_mov_b32 v11, 0
        global_store_dwordx2 v[0:1], v[10:11], off
        buffer_load_dwordx4 v10, s[8:11], 0 offen lds
        s_waitcnt lgkmcnt(0)
        v_mov_b32 v11, 0
        s_endpgm""")
    assert [(x[1], x[2]) for x in h] == [("writes", [11]), ("reads", [10, 11]), ("reads", [10])]


def test_loop_carried_read_and_join(tmp_path):
    # the read issued at the bottom of the loop is still in flight at the top
    # of the next iteration, where it is used before the wait
    h, _ = _hazards(tmp_path, """
        s_mov_b32 s0, 4
        .LBB0_1:
        v_add_u32_e32 v20, v10, v1
        asm: ds_read_b128 v[10:13], v2
        s_add_i32 s0, s0, -1
        s_cmp_lg_u32 s0, 0
        s_cbranch_scc1 .LBB0_1
        s_waitcnt lgkmcnt(0)
        v_mov_b32 v21, v10
        s_endpgm""")
    assert [x[1:] for x in h] == [("reads", [10], "v_add_u32_e32 v20, v10, v1")]
    # on one branch the read is waited for, on the other not: the join keeps it
    h, _ = _hazards(tmp_path, """
        asm: ds_read_b128 v[10:13], v2
        s_cbranch_execz .LBB0_2
        s_waitcnt lgkmcnt(0)
        .LBB0_2:
        v_mov_b32 v21, v12
        s_endpgm""")
    assert [(x[1], x[2]) for x in h] == [("reads", [12])]


def test_library_kernels_have_no_use_before_wait(tmp_path):
    """The GEMM and attention kernels, built with the library's flags."""
    if shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"):
        pytest.skip("hipcc not available")
    r = subprocess.run(["make", "-s", "-C", CSRC, "asm", f"ASMDIR={tmp_path}"],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    total_reads = 0
    for name in ("gemm.s", "attention.s"):
        res, n = chk.check_asm(str(tmp_path / name))
        total_reads += n
        assert res, name
        bad = {k: v[:3] for k, v in res.items() if v}
        assert not bad, f"{name}: {bad}"
    assert total_reads > 100     # the inline-asm reads were seen at all
