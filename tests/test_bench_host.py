"""Host logic of bench.py, without a GPU: the algorithmic bytes each launch is held
to, the kernel-name parsing of rocprofv3 output, the counter summary (calibration,
per-dispatch bytes, rates, traffic.json) and the one-GPU guard."""
import csv
import json
import os
import subprocess
import sys
from types import SimpleNamespace

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def fake_allreduce(nranks, numel, buckets, dtype=0, buf_dtype=0, compress=False, flags=0):
    return SimpleNamespace(nranks=nranks, numel=numel, dtype=dtype, buf_dtype=buf_dtype, compress=compress,
                           tiled_flags=flags,
                           buckets=[SimpleNamespace(tensors=t, count=c, direct=d) for t, c, d in buckets])


def test_kernel_bytes_by_hand():
    # 4 ranks; bucket 0 fuses tensors of 5 and 6 elements into a 12-element buffer (a
    # 16-byte aligned gap of 1); bucket 1 is one direct 100-element tensor
    ar = fake_allreduce(4, [5, 6, 100], [([0, 1], 12, False), ([2], 100, True)])
    kb = lambda kind, b, step=0: bench.kernel_bytes(ar, kind, b, step)  # noqa: E731
    assert kb("pack", 0) == 4 * (4 * 11 + 4 * 12)  # every rank: read its tensors, write its whole buffer
    assert kb("pack_rs", 0) == 4 * 4 * 11 + 3 * 4 * 12  # no sender stores its own sent chunk
    assert kb("rs", 0) == 3 * 4 * 12 and kb("ag", 0) == 2 * 4 * 12 and kb("rs_ag", 0) == 4 * 4 * 12
    assert kb("unpack", 0) == kb("ag_unpack", 0) == 4 * 8 * 11
    assert kb("fold", 0) == 2 * 4 * 4 * 12
    assert kb("rs", 1) == 3 * 4 * 100 and kb("fold", 1) == 2 * 4 * 4 * 100
    # the compressed ring on the direct tensor: binary32 in place, binary16 wire
    arc = fake_allreduce(4, [5, 6, 100], [([0, 1], 12, False), ([2], 100, True)], buf_dtype=1, compress=True)
    kc = lambda kind, b, step=0: bench.kernel_bytes(arc, kind, b, step)  # noqa: E731
    assert kc("rs", 1, 0) == 10 * 100 and kc("rs", 1, 1) == 8 * 100  # first touch reads two binary32 values
    assert kc("rs_ag", 1) == 14 * 100 and kc("ag", 1, 0) == 10 * 100 and kc("ag", 1, 1) == 8 * 100
    assert kc("rs", 0) == 3 * 2 * 12  # the fused buffer is binary16
    assert kc("pack_rs", 0) == 4 * 4 * 11 + 3 * 2 * 12 and kc("ag_unpack", 0) == 4 * 6 * 11


def test_whole_cycle_bytes_match_the_step_count():
    """A fused cycle's launches add up to the separate copy-in, ring and copy-out less
    what fusion saves, in buffer elements: adding step 0's two reads and its write (3),
    the sender copies nothing reads (1), the owner's re-read in the fused middle step
    (1), and the last replacing step's read and write (2)."""
    n, data, count = 8, 1000, 1003
    ar = fake_allreduce(n, [data], [([0], count, False)])
    launches = [("pack_rs", 0)] + [("rs", s) for s in range(1, n - 2)] + [("rs_ag", 0)] \
        + [("ag", s) for s in range(1, n - 2)] + [("ag_unpack", 0)]
    total = sum(bench.kernel_bytes(ar, k, 0, s) for k, s in launches)
    separate = n * (4 * data + 4 * count) + (n - 1) * 5 * 4 * count + n * 8 * data
    assert total == separate - (3 + 1 + 1 + 2) * 4 * count


def test_replacing_into_tensors_bytes():
    """With the replacing steps writing the tensors, the fused step reads two buffers and
    writes two ranks' tensors, a replacing step copies one rank's tensors to the next
    (tensor elements only: padding is not moved), and no copy-out follows: against the
    replacing steps in the buffers the cycle moves 2(N-1) fewer binary32 values per
    buffer element (the copy-out's N reads and N writes, less one replacing step's read
    and write, less the padding the fused step and the replacing steps no longer move)."""
    n, data, count = 8, 1000, 1003
    ar = fake_allreduce(n, [data, 50], [([0], count, False), ([1], 50, True)], flags=bench.TILED_REPLACE_IN_TENSORS)
    assert bench.kernel_bytes(ar, "rs_ag", 0, n - 2) == 4 * 4 * data
    assert bench.kernel_bytes(ar, "ag", 0, 3) == 2 * 4 * data
    assert bench.kernel_bytes(ar, "ag", 1, 3) == 2 * 4 * 50 and bench.kernel_bytes(ar, "rs_ag", 1, n - 2) == 4 * 4 * 50
    launches = [("pack_rs", 0)] + [("rs", s) for s in range(1, n - 2)] + [("rs_ag", n - 2)] \
        + [("ag", s) for s in range(1, n - 1)]
    into = sum(bench.kernel_bytes(ar, k, 0, s) for k, s in launches)
    ab = fake_allreduce(n, [data], [([0], count, False)])
    launches = [("pack_rs", 0)] + [("rs", s) for s in range(1, n - 2)] + [("rs_ag", n - 2)] \
        + [("ag", s) for s in range(1, n - 2)] + [("ag_unpack", n - 2)]
    buffers = sum(bench.kernel_bytes(ab, k, 0, s) for k, s in launches)
    assert buffers - into == 2 * (n - 1) * 4 * count


def test_adding_from_tensors_bytes():
    """With the adding steps reading each receiver's own elements from its tensors as well,
    a cycle moves only the ring's messages: 3 elements per adding step, 4 in the fused step,
    2 per replacing step, each over the tensors' elements (5N-6 per element in all)."""
    n, data, count = 8, 1000, 1003
    flags = bench.TILED_REPLACE_IN_TENSORS | bench.TILED_ADD_FROM_TENSORS
    ar = fake_allreduce(n, [data, 50], [([0], count, False), ([1], 50, True)], flags=flags)
    assert bench.kernel_bytes(ar, "rs", 0, 0) == bench.kernel_bytes(ar, "rs", 0, 3) == 3 * 4 * data
    assert bench.kernel_bytes(ar, "rs", 1, 3) == 3 * 4 * 50  # a direct tensor's ring is not affected
    launches = [("rs", s) for s in range(n - 2)] + [("rs_ag", n - 2)] + [("ag", s) for s in range(1, n - 1)]
    assert sum(bench.kernel_bytes(ar, k, 0, s) for k, s in launches) == (5 * n - 6) * 4 * data


def test_a_launch_serving_two_buckets_counts_both():
    """The same ring step of two fusion buffers in one launch moves both rings' bytes."""
    ar = fake_allreduce(5, [300, 200, 77], [([0], 300, False), ([1, 2], 280, False)])
    for kind in ("rs", "rs_ag", "ag"):
        assert bench.kernel_bytes(ar, kind, (0, 1), 1) == bench.kernel_bytes(ar, kind, 0, 1) + \
            bench.kernel_bytes(ar, kind, 1, 1)
        assert bench.kernel_name(ar, kind, (0, 1)) == bench.kernel_name(ar, kind, 0)
    assert bench.kernel_bytes(ar, "rs", (0, 1), 1) == 3 * 4 * (300 + 280)


REAL_NAMES = {
    "void hvdx::(anonymous namespace)::unpack_kernel<float, float, hvdx::(anonymous namespace)::CopyCfg<2, 2, 2, "
    "true, true, false, 1>, true>(hvdx::RankPtrs, long, void* const*, long const*, long const*, int, int, int, "
    "long, long)": ("ag_unpack", "CopyCfg<2,2,2,true,true,false,1>"),
    "void hvdx::(anonymous namespace)::pack_kernel<float, float, hvdx::(anonymous namespace)::CopyCfg<1, 2, 4, "
    "true, true, false, 1>, false>(void const* const*, long const*, long const*, int, hvdx::RankPtrs, long, int, "
    "int, long, long, int)": ("pack", "CopyCfg<1,2,4,true,true,false,1>"),
    "void hvdx::(anonymous namespace)::rs_step_kernel<float, 0, true, hvdx::(anonymous namespace)::Policy<2, 256, "
    "false, true, false> >(hvdx::RankPtrs, hvdx::RingArgs)": ("rs_step_f32", "Policy<2,256,false,true,false>"),
    "_ZN4hvdx12_GLOBAL__N_118rs_step_c16_kernelILi0ELb0ELb1ENS0_6PolicyILi1ELi64ELb1ELb1ELb0EEEEEvNS_8RankPtrsEPD"
    "F16_NS_8RingArgsE": ("rs_step_c16", "Policy<1,64,1,1,0>"),
    "_ZN4hvdx12_GLOBAL__N_111pack_kernelIfDF16_NS0_7CopyCfgILi2ELi2ELi2ELb1ELb1ELb0ELi1EEELb1EEEvPKPKvPKlS9_iNS_8"
    "RankPtrsEliilli": ("pack_rs", "CopyCfg<2,2,2,1,1,0,1>"),
    "_ZN4hvdx12_GLOBAL__N_114ag_step_kernelIDF16_Lb1ENS0_6PolicyILi2ELi512ELb0ELb0ELb0EEEEEvNS_8RankPtrsENS_8Ring"
    "ArgsE": ("ag_step_f16", "Policy<2,512,0,0,0>"),
    "_ZN4hvdx12_GLOBAL__N_121rs_ag_step_c16_kernelILi1ELb0ELb1ENS0_6PolicyILi1ELi64ELb1ELb1ELb0EEEEEvNS_8RankPtrs"
    "EPKDF16_NS_8RingArgsE": ("rs_ag_step_c16", "Policy<1,64,1,1,0>"),
    "void hvdx::(anonymous namespace)::small_cycle_kernel<float, float, 1>(void const* const*, long const*, long "
    "const*, int, hvdx::RankPtrs, hvdx::RingArgs, long)": ("cycle_small", ""),
    "void hvdx::(anonymous namespace)::rs_ag_step_pair_kernel<float, 1, true, hvdx::(anonymous namespace)::Policy<1, "
    "256, false, true, false> >(hvdx::RingPair)": ("rs_ag_step_f32", "Policy<1,256,false,true,false> x2"),
    "void hvdx::(anonymous namespace)::ag_step_pair_kernel<float, true, hvdx::(anonymous namespace)::Policy<2, 512, "
    "false, true, false> >(hvdx::RingPair)": ("ag_step_f32", "Policy<2,512,false,true,false> x2"),
    "void hvdx::(anonymous namespace)::unpack_pair_kernel<float, float, hvdx::(anonymous namespace)::CopyCfg<2, 1, 2, "
    "true, true, false, 1, 256> >(hvdx::CopyPair, int, int, int)": ("ag_unpack", "CopyCfg<2,1,2,true,true,false,1,256> x2"),
    "_ZN4hvdx12_GLOBAL__N_116pack_pair_kernelIfDF16_NS0_7CopyCfgILi2ELi2ELi2ELb1ELb1ELb0ELi1ELi256EEEEEvNS_8CopyPairEiii":
        ("pack_rs", "CopyCfg<2,2,2,1,1,0,1,256> x2"),
    "void hvdx::(anonymous namespace)::pack_tiles_kernel<float, float, 1>(hvdx::TiledCopy, int)": ("pack_rs", "tiles<1>"),
    "void hvdx::(anonymous namespace)::unpack_tiles_kernel<float, float, 1>(hvdx::TiledCopy, int)":
        ("ag_unpack", "tiles<1>"),
    "_ZN4hvdx12_GLOBAL__N_117pack_tiles_kernelIfDF16_Li2EEEvNS_9TiledCopyEi": ("pack_rs", "tiles<2>"),
    "_ZN4hvdx12_GLOBAL__N_119unpack_tiles_kernelIfDF16_Li2EEEvNS_9TiledCopyEi": ("ag_unpack", "tiles<2>"),
    "void hvdx::(anonymous namespace)::rs_ag_tiles_kernel<float, float, 2, true, 1>(hvdx::TiledCopy, "
    "hvdx::RingArgs)": ("rs_ag_step_f32", "tiles<1>"),
    "void hvdx::(anonymous namespace)::ag_tiles_kernel<float, false, 2, 1>(hvdx::TiledCopy, int, int, long)":
        ("ag_step_f32", "tiles<1>"),
    "_ZN4hvdx12_GLOBAL__N_115ag_tiles_kernelIDF16_Lb1ELi2ELi1EEEvNS_9TiledCopyEiil": ("ag_step_f16", "tiles<1>"),
    "void hvdx::(anonymous namespace)::add_tiles_kernel<float, float, true, 2, 1>(hvdx::TiledCopy, int, int, long)":
        ("rs_step_f32", "tiles<1>"),
    "_ZN4hvdx12_GLOBAL__N_116add_tiles_kernelIfDF16_Lb0ELi2ELi2EEEvNS_9TiledCopyEiil": ("rs_step_c16", "tiles<2>"),
    "_ZN4hvdx12_GLOBAL__N_118rs_ag_tiles_kernelIfDF16_Li2ELb1ELi2EEEvNS_9TiledCopyENS_8RingArgsE":
        ("rs_ag_step_c16", "tiles<2>"),
    "__amd_rocclr_copyBuffer": (None, ""),
}


@pytest.mark.parametrize("name", list(REAL_NAMES))
def test_kernel_names_from_rocprof(name):
    short, shape = REAL_NAMES[name]
    assert bench.short_kernel_name(name) == short
    assert bench.shape_of(name) == shape


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_summarize_profiles_scales_counters_by_the_copy(tmp_path, monkeypatch):
    """FETCH_SIZE reads half of what a plain 1 GiB copy moves and WRITE_SIZE all of it:
    factors 2 and 1.  A kernel counted at 100 KiB fetched and 50 KiB written per
    dispatch, 1 us on average, moves 256,000 bytes at 256 GB/s."""
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    d = tmp_path / "out"
    rs = list(REAL_NAMES)[2]
    _write_csv(str(d / "prof_w" / "w_kernel_stats.csv"), ["Name", "Calls", "TotalDurationNs"],
               [[rs, 10, 10_000], ["__amd_rocclr_copyBuffer", 3, 1_000_000]])
    hdr = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    _write_csv(str(d / "pmc_fetch_w" / "fetch_counter_collection.csv"), hdr,
               [["__amd_rocclr_copyBuffer", 1 << 20, "FETCH_SIZE", 1 << 19]] * 3
               + [[rs, 4096, "FETCH_SIZE", 100.0]] * 2)
    _write_csv(str(d / "pmc_write_w" / "write_counter_collection.csv"), hdr,
               [["__amd_rocclr_copyBuffer", 1 << 20, "WRITE_SIZE", 1 << 20]] * 3
               + [[rs, 4096, "WRITE_SIZE", 50.0]] * 2)
    text = bench.summarize_profiles(str(d))
    assert "FETCH_SIZE x 2.000 and WRITE_SIZE x 1.000" in text
    row = [line for line in text.splitlines() if line.startswith("| rs_step_f32")]
    assert row == ["| rs_step_f32 | `Policy<2,256,false,true,false>` | 10 | 1.00 | 0.01 | 0.2 | 0.1 | 256 | 3.2 |",
                   "| rs_step_f32 | 10 | 1.00 | 0.01 | 0.3 |"]  # the per-reported-kernel table
    rec = json.load(open(tmp_path / "traffic.json"))
    assert rec["per_launch_bytes"] == {"w/rs_step_f32": 256000}
    assert rec["calibration"] == {"w": {"FETCH_SIZE": 2.0, "WRITE_SIZE": 1.0}}
    assert rec["source_hash"] == bench.kernel_source_hash()


def test_bench_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_fusion_buffer_modes_are_fused_allreduce_arguments():
    import inspect

    from paper_1802_05799_amd import cycle

    params = inspect.signature(cycle.FusedAllreduce.__init__).parameters
    assert bench.BUFFER_MODES["ring_on_tensors"] == {}
    for mode in bench.BUFFER_MODES.values():
        assert all(k in params and params[k].default is True for k in mode) and all(v is False for v in mode.values())
