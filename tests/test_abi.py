"""The C interface on the CPU: the library loads, exports every declared
entry point, and its host-side validation and record layout behave as
specified (no device work is issued by these calls)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LC.LIB_PATH):
        from paper_2609_27193_amd.build_lib import build
        build()
    return LC.load_library()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "layercheck.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lc_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(LC.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


FAKE = 0x7F0000000000  # never dereferenced by lc_query_layout


def fake_segments(sizes, esz=2, master=True, offset=0, moments=True):
    segs, addr = [], FAKE + offset
    for l, layer in enumerate(sizes):
        for n in layer:
            step = (n * 4 + 255) // 256 * 256
            segs.append(LC.Segment(l, n, addr, addr + step, addr + 2 * step if master else None,
                                   addr + 3 * step if moments else None, addr + 4 * step if moments else None))
            addr += 5 * step
    return segs


def desc(segs, n_layers, **kw):
    args = dict(weight_dtype=LC.LC_DT_BF16, has_master=True, mode=LC.LC_MODE_ACCUM,
                k0=[1e-3] * n_layers, s_max=8, eps_w=1e-8, t_base=0)
    args.update(kw)
    return LC.LayoutDesc(segs, n_layers, **args)


@pytest.mark.parametrize("sizes,dtype,master", [
    ([[1], [3, 7], [8, 1023, 4097]], LC.LC_DT_BF16, True),
    ([[65536 * 3 + 5], [128]], LC.LC_DT_BF16, False),
    ([[17, 33], [100000]], LC.LC_DT_F32, False),
])
def test_record_bytes_match_oracle(lib, sizes, dtype, master):
    segs = fake_segments(sizes, esz=2 if dtype == LC.LC_DT_BF16 else 4, master=master)
    numel, rec = LC.lc_query_layout(desc(segs, len(sizes), weight_dtype=dtype, has_master=master))
    assert numel == [sum(l) for l in sizes]
    esz = 2 if dtype == LC.LC_DT_BF16 else 4
    assert rec == [O.record_bytes(l, esz, master) for l in sizes]


@pytest.mark.parametrize("master", [True, False])
def test_weights_only_records_match_oracle(lib, master):
    """The SGD variant (Section 4.7): records hold the weights (and master)
    without Adam moments."""
    sizes = [[4097, 5], [128]]
    segs = fake_segments(sizes, master=master, moments=False)
    _, rec = LC.lc_query_layout(desc(segs, 2, has_master=master))
    assert rec == [O.record_bytes(l, 2, master, has_moments=False) for l in sizes]
    assert O.record_bytes([128], 2, True, has_moments=False) == 6 * 128
    mixed = fake_segments(sizes, master=master, moments=False)
    mixed[1].exp_avg = FAKE + (1 << 30)
    with pytest.raises(LC.LCError):
        LC.lc_query_layout(desc(mixed, 2, has_master=master))


def _expect(code, fn):
    with pytest.raises(LC.LCError) as e:
        fn()
    assert e.value.code == code, str(e.value)
    assert LC.load_library().lc_last_error().decode()


def test_validation_errors(lib):
    good = fake_segments([[4], [4]])
    q = lambda **kw: LC.lc_query_layout(desc(kw.pop("segs", good), kw.pop("n", 2), **kw))
    q()  # valid
    I = LC.LC_ERR_INVALID_ARG
    _expect(I, lambda: q(weight_dtype=3))
    _expect(I, lambda: q(mode=2))
    _expect(I, lambda: q(s_max=0))
    _expect(I, lambda: q(eps_w=-1.0))
    _expect(I, lambda: q(eps_w=float("inf")))
    _expect(I, lambda: q(k0=[1e-3, -1.0]))
    _expect(I, lambda: q(k0=[1e-3, float("nan")]))
    _expect(I, lambda: q(has_master=False))         # master pointers present
    _expect(I, lambda: q(segs=good[::-1]))            # not grouped by ascending layer
    _expect(I, lambda: q(n=3, k0=[1e-3] * 3))         # layer 2 has no segment
    bad = fake_segments([[4], [4]])
    bad[0].numel = 0
    _expect(I, lambda: q(segs=bad))
    bad = fake_segments([[4], [4]])
    bad[1].weight += 1                                  # odd address for bf16
    _expect(I, lambda: q(segs=bad))
    bad = fake_segments([[4], [4]])
    bad[1].shadow = bad[1].weight
    _expect(I, lambda: q(segs=bad))
    bad = fake_segments([[4], [4]])
    bad[0].exp_avg = 0
    _expect(I, lambda: q(segs=bad))
    bad = fake_segments([[4], [4]])
    bad[1].layer = 5
    _expect(I, lambda: q(segs=bad))
    # no two arrays may share a byte, within a segment or across segments
    for a, b, shift in [(0, 0, 0), (1, 0, 0), (1, 0, 4), (0, 0, -4)]:
        bad = fake_segments([[4], [4]])
        bad[a].exp_avg_sq = bad[b].exp_avg + shift       # v on (or straddling) another segment's m
        _expect(I, lambda: q(segs=bad))
        assert "overlap" in lib.lc_last_error().decode()
    bad = fake_segments([[4], [4]])
    bad[1].master = bad[0].weight + 4                   # fp32 master over the tail of a bf16 weight
    _expect(I, lambda: q(segs=bad))
    # arrays that touch without overlapping are fine
    a = FAKE
    tight = [LC.Segment(0, 4, a, a + 8, a + 16, a + 32, a + 48), LC.Segment(1, 4, a + 64, a + 72, a + 80, a + 96, a + 112)]
    q(segs=tight)
    big = fake_segments([[1 << 40]])
    _expect(I, lambda: q(segs=big, n=1, k0=[1e-3], s_max=1 << 30))  # staleness numerator overflow
    # element counts are bounded before any byte count is formed from them
    huge = fake_segments([[1 << 46] * 65])
    _expect(I, lambda: q(segs=huge, n=1, k0=[1e-3]))
    assert "too many elements" in lib.lc_last_error().decode()
    huge = fake_segments([[1 << 46] * 64] * 17)
    _expect(I, lambda: q(segs=huge, n=17, k0=[1e-3] * 17))
    assert "too many elements" in lib.lc_last_error().decode()
    with pytest.raises(ValueError):
        desc(good, 2, k0=[1e-3])


def test_null_handling(lib):
    assert lib.lc_destroy(None) == LC.LC_OK
    assert lib.lc_record_bytes(None, 0) == 0
    assert lib.lc_query_layout(None, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_init_layout(None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_score_layers(None, 1) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_select(None, 1, 1.0, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_pack_selected(None, None, 0, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_read_state(None, None, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_restore_composite(None, None, 0, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_rebase(None, 1) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_adamw_step_score(None, 1, None, LC.LC_DT_BF16, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_sgd_step_score(None, 1, None, LC.LC_DT_BF16, None, None) == LC.LC_ERR_INVALID_ARG
    # the store: NULL handles and arguments are refused, closing NULL is a no-op
    assert lib.lc_store_open(None, 1, None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_append(None, 0, None, None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_append_async(None, 0, None, None, 0, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_sync(None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_count(None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_entry(None, 0, None, None, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_plan(None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_restore(None, None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_compact(None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_discard_after(None, 0, None) == LC.LC_ERR_INVALID_ARG
    assert lib.lc_store_close(None) == LC.LC_OK
    assert lib.lc_last_error()  # the last refusal's message


def test_invalid_init_enqueues_nothing(lib):
    # validation happens before any HIP call, so this runs without a GPU
    bad = fake_segments([[4], [4]])
    bad[0].numel = 0
    _expect(LC.LC_ERR_INVALID_ARG, lambda: LC.lc_init_layout(desc(bad, 2)))


def test_missing_library_fails_loudly(tmp_path):
    """No fallback: without the built library the binding refuses to run."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("from paper_2609_27193_amd import layercheck as LC\n"
            "try:\n    LC.load_library()\nexcept RuntimeError as e:\n    print('refused:', e)\n")
    env = dict(os.environ, LAYERCHECK_LIB=str(tmp_path / "absent.so"), PYTHONPATH=root)
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "refused:" in out.stdout and "not built" in out.stdout


def test_struct_layouts_match_header(tmp_path):
    """The binding's ctypes structures have the C compiler's layout of the
    header's structures: every size and member offset, from a probe compiled
    against include/layercheck.h."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc") or shutil.which("cc")
    if gcc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    structs = {"lc_segment": LC.lc_segment, "lc_layout_desc": LC.lc_layout_desc,
               "lc_select_stats": LC.lc_select_stats, "lc_pack_result": LC.lc_pack_result,
               "lc_version": LC.lc_version, "lc_adamw_params": LC.lc_adamw_params,
               "lc_sgd_params": LC.lc_sgd_params}
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "layercheck.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} size %zu\\n", sizeof({name}));')
        for field, _ in cls._fields_:
            lines.append(f'  printf("{name} {field} %zu\\n", offsetof({name}, {field}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([gcc, "-std=c11", "-I", os.path.join(root, "include"), "-o", str(exe), str(src)], check=True,
                   capture_output=True, timeout=120)
    got = {}
    for line in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines():
        name, key, value = line.split()
        got[(name, key)] = int(value)
    for name, cls in structs.items():
        assert got[(name, "size")] == C.sizeof(cls), name
        for field, _ in cls._fields_:
            assert got[(name, field)] == getattr(cls, field).offset, (name, field)


def test_init_refuses_memory_hip_does_not_know(lib):
    """The device-range check runs before anything is allocated or enqueued:
    arrays that are not device memory (here, addresses no GPU allocation
    holds) are refused with LC_ERR_INVALID_ARG, so the call needs no GPU."""
    segs = fake_segments([[4], [4]])
    with pytest.raises(LC.LCError) as e:
        LC.lc_init_layout(desc(segs, 2))
    assert e.value.code == LC.LC_ERR_INVALID_ARG
    assert "not device memory" in lib.lc_last_error().decode()


def test_build_info(lib):
    info = LC.lc_query_build()
    assert info["record_align"] == 256
    assert info["chunk_bytes"] % (16 * 256) == 0 and info["piece_bytes"] % (16 * 256) == 0


def test_reduced_layouts_span_tiles(lib):
    """The reduced layouts of the GPU parity tests reach every kernel path at
    the tile sizes this build reports: for each array, some tensor spans full
    tiles and ends in a ragged one (score chunks over the weights; pack and
    restore pieces over the weights, master and moments), and some tensor is
    smaller than one tile."""
    from paper_2609_27193_amd import inputs as I
    from tests.test_parity_gpu import reduced_13b, reduced_8b, reduced_qwen, tied_spec
    info = LC.lc_query_build()
    for spec in (reduced_8b(), reduced_qwen(), reduced_13b(), tied_spec()):
        sizes = [t.numel for l in spec.layers for t in l.tensors]
        w = spec.weight_bytes
        arrays = [("weight", w, (info["chunk_bytes"], info["piece_bytes"]))]
        arrays += [(a, 4, (info["piece_bytes"],)) for a in (["master"] if spec.has_master else [])
                   + ["exp_avg", "exp_avg_sq"]]
        for name, esz, tiles in arrays:
            for tile in tiles:
                nbytes = [n * esz for n in sizes]
                assert any(b > tile and b % tile for b in nbytes), (spec.name, name, tile)
                assert any(b < tile for b in nbytes), (spec.name, name, tile)
                assert sum(b // tile for b in nbytes) >= 8, (spec.name, name, tile)


def test_static_score_refuses_before_any_device_work(lib):
    """lc_score_layers_static checks its arguments and sizes on the host before
    it touches the GPU: a layer whose tables exceed the fixed device array is
    refused with LC_ERR_CAPACITY, malformed lists with LC_ERR_INVALID_ARG."""
    big = fake_segments([[1 << 30], [4_000_000_000]])  # 4e9 bf16 weights: ~19 MB of chunk tables
    u = 0x7E0000000000

    def status(segs, n_layers, dtype=LC.LC_DT_BF16, u_out=u):
        arr = (LC.lc_segment * len(segs))()
        for i, s in enumerate(segs):
            arr[i] = LC.lc_segment(s.layer, 0, s.numel, s.weight, s.shadow, None, None, None)
        return lib.lc_score_layers_static(arr, len(segs), n_layers, dtype, 1e-8, u_out, None)

    assert status(big, 2) == LC.LC_ERR_CAPACITY
    assert b"layer 1" in LC.load_library().lc_last_error()
    assert status(big, 3) == LC.LC_ERR_INVALID_ARG        # layer 2 has no segment
    assert status(big[::-1], 2) == LC.LC_ERR_INVALID_ARG  # not grouped by ascending layer
    assert status(big, 2, dtype=5) == LC.LC_ERR_INVALID_ARG
    assert status(big, 2, u_out=None) == LC.LC_ERR_INVALID_ARG
