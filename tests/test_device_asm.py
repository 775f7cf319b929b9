"""Checks on the gfx950 assembly of the library's own kernels (no GPU).

The device code is compiled to assembly (hipcc -S, device pass only) and
scanned for properties the kernels rely on:
  * no store through a buffer descriptor uses a register soffset: the
    compiler then treats the store's data registers as free for the next
    VALU write, which corrupted outputs on gfx950; with a constant soffset it
    inserts the wait states;
  * no store of more than 64 bits is followed directly by a VALU write of its
    data registers;
  * no kernel spills to scratch (and the benchmark workloads' kernels are
    checked by name);
  * the reductions use DPP and the gfx950 permlane swaps, the exponentials
    v_exp_f32, and bf16 outputs v_cvt_pk_bf16_f32;
  * row loads are non-temporal and row stores non-temporal, at device scope
    only where a launch's stores cover whole 128-byte lines.
"""
import os
import re
import subprocess

import pytest

from paper_2607_23089_amd import build as B


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    from concurrent.futures import ThreadPoolExecutor
    d = tmp_path_factory.mktemp("asm")

    def one(src):
        out = d / (os.path.basename(src) + ".s")
        cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only",
               "-S", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", B.INCLUDE, "-I", B.CSRC, "-o", str(out), src]
        subprocess.run(cmd, check=True, capture_output=True)
        return out.read_text()

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as pool:
        return "\n".join(pool.map(one, B.SOURCES))


def kernels(asm):
    return {m.group(1): m.group(2) for m in
            re.finditer(r"\.amdhsa_kernel (\S+)(.*?)\.end_amdhsa_kernel", asm, re.S)}


def test_buffer_stores_use_constant_soffset(asm):
    soffs = re.findall(r"buffer_store_\S+ \S+, \S+, s\[\d+:\d+\], (\S+)", asm)
    assert soffs, "no buffer stores found"
    assert set(soffs) == {"0"}


def test_no_immediate_overwrite_of_store_data(asm):
    lines = asm.splitlines()
    for i, line in enumerate(lines):
        m = re.match(r"\s*(?:buffer|global)_store_dwordx(?:3|4) v\[(\d+):(\d+)\]", line)
        if not m:
            m2 = re.match(r"\s*global_store_dwordx(?:3|4) \S+, v\[(\d+):(\d+)\]", line)
            if not m2:
                continue
            m = m2
        lo, hi = int(m.group(1)), int(m.group(2))
        nxt = lines[i + 1].strip()
        d = re.match(r"v_\S+\s+v(\d+)", nxt)
        assert not (d and lo <= int(d.group(1)) <= hi), f"{line.strip()} | {nxt}"


@pytest.mark.parametrize("pattern", [
    # template arguments: ..., output form (0 softmax, 1 fused, 2 log)
    r"small_row_kernelINS_4BF16ES1_Li8ELi8ELi4ELi0E",      # small_262144x64
    r"medium_row_kernelINS_4BF16ES1_Li8ELi2ELb0ELi0E",     # causal_32768x4096
    r"medium_row_kernelINS_3F32ES1_Li4ELi4ELb0ELi0E",      # fp32_64x1000
    r"split_row_kernelINS_4BF16ENS_3F32ELi4ELi10ELi0ELb0E",    # vocab_4096x151936
    r"split_row_kernelINS_3F32ES1_Li4ELi16ELi0ELb0E",          # large_1024x262144
    r"large_row_kernelINS_3F32ES1_Li4ELi4ELi0E",           # two-pass form
    r"medium_row_kernelINS_4BF16ES1_Li8ELi2ELb0ELi1E",     # fused causal 32768x4096
    r"split_row_kernelINS_3F32ES1_Li4ELi8ELi1ELb0E",           # fused f32 long rows
    r"small_row_kernelINS_4BF16ES1_Li8ELi8ELi4ELi1E",      # fused small rows
    r"split_row_kernelINS_4BF16ENS_3F32ELi4ELi10ELi2ELb0E",    # log-softmax vocab_4096x151936
    r"split_row_kernelINS_3F32ES1_Li4ELi16ELi2ELb0E",          # log-softmax 1024x262144
    r"medium_row_kernelINS_4BF16ES1_Li8ELi19ELb1ELi2E",    # log-softmax packed bf16 151936
    r"medium_row_kernelINS_4BF16ES1_Li8ELi2ELb0ELi2E",     # log-softmax 4096-wide rows
    r"bwd_small_kernelINS_4BF16ES1_Li8ELi8ELi4EEE",        # bwd_small_262144x64
    r"bwd_medium_kernelINS_4BF16ES1_Li8ELi2EEE",           # bwd_causal_32768x4096
    r"bwd_split_kernelINS_3F32ES1_Li4ELi8EEE",             # bwd_large_1024x262144
    r"bwd_large_kernelINS_3F32ES1_Li4ELi4EEE",             # backward two-pass form
    r"group_top2_kernelINS_3F32ES1_Li4ELi8ELi4EEE",        # moe_*x256_f32, groups of 32
    r"group_top2_kernelINS_4BF16ENS_3F32ELi8ELi4ELi4EEE",  # moe_65536x256_bf16
])
def test_workload_kernels_do_not_spill(asm, pattern):
    ks = {k: v for k, v in kernels(asm).items() if re.search(pattern, k)}
    assert len(ks) == 1, pattern
    body = next(iter(ks.values()))
    assert int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", body).group(1)) == 0


def test_no_kernel_spills(asm):
    # every instantiation the launchers can choose keeps its data in registers
    spills = {k: int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", v).group(1))
              for k, v in kernels(asm).items()}
    assert spills, "no kernels found"
    bad = {k: v for k, v in spills.items() if v}
    assert not bad, f"{len(bad)} kernels spill, e.g. {sorted(bad.items())[:3]}"


def test_split_exchange_has_no_cache_maintenance(asm):
    # The exchange words are self-validating 64-bit atomics: no L2 write-back
    # or invalidation may appear in the split kernel (each one serialises the
    # whole device), and the polls and stores are device-coherent (sc1).
    body = asm[asm.index("split_row_kernelINS_3F32ES1_Li4ELi16ELi0E"):]
    body = body[:body.index("s_endpgm")]
    assert "buffer_wbl2" not in body and "buffer_inv" not in body
    assert "s_sleep" in body
    assert re.search(r"global_store_dwordx2 .* sc1", body)
    assert re.search(r"global_load_dwordx2 .* sc1", body)


def test_expected_instructions(asm):
    for ins in ("row_half_mirror", "row_mirror", "quad_perm:[1,0,3,2]",
                "v_permlane16_swap_b32", "v_permlane32_swap_b32", "v_exp_f32",
                "v_cvt_pk_bf16_f32", "buffer_load_dwordx4", "buffer_store_dwordx4",
                "v_log_f32", "v_maximum3_f32", "v_minimum3_f32"):
        assert ins in asm, ins
    # no packed-fp32 arithmetic anywhere
    assert not re.search(r"v_pk_(add|mul|fma)_f32", asm)


def test_stream_cache_policy(asm):
    # row data streams through: loads non-temporal; stores non-temporal, at
    # device scope only where the launch's stores cover whole 128-byte lines
    # (each store site has both forms behind a uniform branch), never at
    # device scope in the ragged and flat kernels, whose rows never start on
    # lines
    stores = re.findall(r"buffer_store_(?:dword|short)\S* .*", asm)
    loads = re.findall(r"buffer_load_(?:dword|ushort)\S* .*", asm)
    assert stores and loads
    assert all(re.search(r" nt( sc1)?$", st) for st in stores), \
        [st for st in stores if not re.search(r" nt( sc1)?$", st)][:3]
    assert all(re.search(r" nt$", ld) for ld in loads), \
        [ld for ld in loads if not re.search(r" nt$", ld)][:3]
    bodies = kernel_bodies(asm)
    checked = 0
    for n, body in bodies.items():
        st = re.findall(r"buffer_store_(?:dword|short)\S* .*", body)
        if not st:
            continue
        dev = sum(bool(re.search(r" nt sc1$", x)) for x in st)
        if re.search(r"ragged_row_kernel|flat_row_kernel|bwd_flat_kernel", n):
            assert dev == 0, n
        elif re.search(r"(small|medium|split|large)_row_kernel|bwd_\w+_kernel", n):
            assert 0 < dev < len(st), (n, dev, len(st))
            checked += 1
    assert checked > 100, checked


def kernel_bodies(asm):
    return {m.group(1): m.group(2) for m in
            re.finditer(r"^(_ZN5rowsm\S*):[^\n]*\n(.*?)\.Lfunc_end", asm, re.S | re.M)}


def serialised_loads(body):
    """Row loads followed by a wait for every load in flight before the next
    row load is issued, and the number of row loads."""
    lines = [ln.strip() for ln in body.splitlines()]
    loads = serial = 0
    for i, ln in enumerate(lines):
        if ln.startswith("buffer_load"):
            loads += 1
            for nxt in lines[i + 1:i + 12]:
                if nxt.startswith("buffer_load"):
                    break
                if nxt.startswith("s_waitcnt") and "vmcnt(0)" in nxt:
                    serial += 1
                    break
    return serial, loads


def test_one_element_bf16_loads_stay_in_flight_together(asm):
    # rows of bf16 that take one-element (2-byte) vectors: the per-slot
    # loads of the medium, small, single-read and MoE kernels are all issued
    # before the first wait, not one memory round trip per slot (a load in a
    # branch had its widening sunk into the branch, with a wait for each)
    # (kernels with at least 4 slots: NV of the medium and single-read
    # forms, row groups per lane of the small and MoE forms)
    bodies = kernel_bodies(asm)
    checked = 0
    for n, body in bodies.items():
        m = re.match(r"_ZN5rowsm(17medium_row|16split_row|16small_row|17group_top2)_kernelINS_4BF16E"
                     r"(?:NS_3F32E|S1_)Li1ELi(\d+)E(?:Li(\d+)E)?", n)
        if not m:
            continue
        slots = int(m.group(2) if m.group(1) in ("17medium_row", "16split_row") else m.group(3))
        if slots < 4:
            continue
        serial, loads = serialised_loads(body)
        checked += 1
        assert serial <= loads // 2, (n, serial, loads)
    assert checked > 100, checked
