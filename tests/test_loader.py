"""Range-read reload source (Sec. IV loader), on the CPU.

The library opens safetensors files and fills the plan's packed weight
inflow buffer with only the byte intervals the plan needs.  The files are
written by the safetensors package itself (an independent writer) from the
seeded content, and the loaded bytes must equal the oracle's packed inflow,
byte for byte.  Error paths (missing or mismatched tensors, truncated or
malformed files) must be rejected with ATP_EINVAL.
"""
import ctypes as C
import json
import random

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import model, repack
from paper_2511_11617_amd import atp, problem
from synth import checkpoint, configs, pagetable
from synth.content import KIND_TAG16, Content
from tests.test_oracle_repack import tiny_cfg


def _tensors(c):
    tl = problem.tensor_list(c)
    return [(n, l, r, cc) for (n, l, k, sp, r, cc, u) in tl], [checkpoint.name(n, l) for (n, l, *_) in tl]


def _plan(c, flags=0):
    table, pool = pagetable.make_for(c)
    live = repack.live_blocks(table)
    return problem.build(c, n_live=len(live), pool=pool, flags=flags, staging_cap=c.get("staging_cap") or 0).plan()


def _write(c, tmp_path, n_files=1, dtype="bf16"):
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    tens, names = _tensors(c)
    paths = []
    for i in range(n_files):
        p = str(tmp_path / f"model-{i:05d}.safetensors")
        checkpoint.write_package(p, content, tens[i::n_files], dtype)
        paths.append(p)
    return content, paths, names


def _load(plan, paths, names, threads=0):
    st = plan.stats()
    buf = np.full(max(st.inflow_w, 1), 0xA5, np.uint8)
    files = atp.StFiles(paths)
    try:
        ls = plan.load_weights(files, names, buf.ctypes.data, st.inflow_w, threads)
    finally:
        files.close()
    return buf[:st.inflow_w], ls


def _check(c, tmp_path, n_files=1, flags=0, dtype="bf16", threads=0, variant="cm"):
    content, paths, names = _write(c, tmp_path, n_files, dtype)
    plan = _plan(c, flags)
    got, ls = _load(plan, paths, names, threads)
    pb = model.build(c, variant=variant)
    want = repack.packed_weight_inflow(pb, content)
    assert got.size == want.size
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {want.size} inflow bytes differ"
    assert ls.bytes == want.size
    return ls


def test_cfg1_fp16_one_column_units(tmp_path):
    # 1-column FFN units make W_down's inflow one 2-byte interval per row
    ls = _check(configs.get(1, w_kind=KIND_TAG16), tmp_path, dtype="fp16")
    assert ls.reads > 0 and ls.bytes < ls.tensor_bytes


@pytest.mark.parametrize("n_files", [2, 3])
def test_tensors_split_over_files(tmp_path, n_files):
    _check(configs.get(1, w_kind=KIND_TAG16), tmp_path, n_files=n_files, threads=3)


@pytest.mark.parametrize("flags,variant", [(atp.PLAN_GREEDY, "greedy"), (atp.PLAN_FULL, "full")])
def test_planner_variants(tmp_path, flags, variant):
    _check(configs.get(1, w_kind=KIND_TAG16), tmp_path, flags=flags, variant=variant)


@settings(max_examples=25, deadline=None)
@given(st.integers(0, 2 ** 31), st.booleans(), st.integers(1, 3), st.integers(1, 4))
def test_random_small(tmp_path_factory, seed, experts, n_files, threads):
    c = tiny_cfg(random.Random(seed), experts)
    _check(c, tmp_path_factory.mktemp("ck"), n_files=n_files, threads=threads)


def test_find_matches_package_data(tmp_path):
    from safetensors import safe_open
    c = configs.get(1, w_kind=KIND_TAG16)
    content, paths, names = _write(c, tmp_path, n_files=2)
    files = atp.StFiles(paths)
    raw = [open(p, "rb").read() for p in paths]
    for nm in names[:6]:
        fi, eb, shape, off, nbytes = files.find(nm)
        with safe_open(paths[fi], "pt") as f:
            t = f.get_tensor(nm)
        assert eb == 2 and shape == tuple(t.shape)
        assert raw[fi][off:off + nbytes] == t.view(dtype=__import__("torch").int16).numpy().tobytes()
    with pytest.raises(atp.AtpError) as e:
        files.find("no.such.tensor")
    assert e.value.code == atp.EINVAL
    files.close()


def test_sparse_stream_writer_holds_the_read_intervals(tmp_path):
    # the full-size benchmark writes only what the plan reads; the loaded
    # bytes must not touch the holes
    c = configs.get(1, w_kind=KIND_TAG16)
    content = Content(c["seed"], c["w_kind"], c["kv_kind"])
    tens, names = _tensors(c)
    plan = _plan(c)
    tl = problem.tensor_list(c)
    regions = []
    for s in plan.segments(atp.SEG_INFLOW_W):
        n, l, kind, sp, rows, cols, unit = tl[s.tensor]
        full = checkpoint.full_words(content, n, l, rows, cols)
        a, b = s.unit_begin * unit, s.unit_end * unit
        if kind == atp.ROWS:
            regions.append((n, l, cols, a, b, 0, cols, full[a:b]))
        else:
            regions.append((n, l, cols, 0, rows, a, b, full[:, a:b]))
    p = str(tmp_path / "sparse.safetensors")
    checkpoint.write_stream(p, tens, regions, "fp16")
    got, _ = _load(plan, [p], names)
    want = repack.packed_weight_inflow(model.build(c), content)
    np.testing.assert_array_equal(got, want)


# ---- error paths ---------------------------------------------------------------

def _expect_einval(fn, match):
    with pytest.raises(atp.AtpError) as e:
        fn()
    assert e.value.code == atp.EINVAL
    assert match in str(e.value), str(e.value)


def _raw(tmp_path, header: bytes, data: bytes = b"", name="bad.safetensors"):
    p = tmp_path / name
    p.write_bytes(len(header).to_bytes(8, "little") + header + data)
    return str(p)


def test_missing_and_mismatched_tensors(tmp_path):
    c = configs.get(1, w_kind=KIND_TAG16)
    content, paths, names = _write(c, tmp_path)
    plan = _plan(c)
    n_in = plan.stats().inflow_w
    buf = np.zeros(n_in, np.uint8)
    files = atp.StFiles(paths)
    _expect_einval(lambda: plan.load_weights(files, names[:-1], buf.ctypes.data, n_in), "one tensor name")
    _expect_einval(lambda: plan.load_weights(files, names[:-1] + ["x"], buf.ctypes.data, n_in), "in none of the files")
    swapped = list(names)
    swapped[0], swapped[1] = swapped[1], swapped[0]   # wq <-> wk: other shape
    _expect_einval(lambda: plan.load_weights(files, swapped, buf.ctypes.data, n_in), "shape")
    _expect_einval(lambda: plan.load_weights(files, names, buf.ctypes.data, n_in - 2), "exactly")
    # the pipelined reload checks the same before any read or GPU work starts
    no_gpu = (None, 0, None, 0)
    _expect_einval(lambda: plan.load_reshard_weights(files, names[:-1], 0, 0, 0, 0, buf.ctypes.data, n_in,
                                                     *no_gpu, None, None), "one tensor name")
    _expect_einval(lambda: plan.load_reshard_weights(files, swapped, 0, 0, 0, 0, buf.ctypes.data, n_in,
                                                     *no_gpu, None, None), "shape")
    # and so does the asynchronous one; nothing is pending after the refusal
    _expect_einval(lambda: plan.load_reshard_weights_async(files, names[:-1], 0, 0, 0, 0, buf.ctypes.data, n_in,
                                                           *no_gpu, None, None), "one tensor name")
    _expect_einval(lambda: plan.load_reshard_weights_async(files, swapped, 0, 0, 0, 0, buf.ctypes.data, n_in,
                                                           *no_gpu, None, None), "shape")
    with pytest.raises(atp.AtpError) as e:
        plan.load_stats()
    assert e.value.code == atp.ESTATE
    files.close()
    # same shapes, 4-byte elements
    tens, _ = _tensors(c)
    import torch
    from safetensors.torch import save_file
    save_file({checkpoint.name(n, l): torch.zeros(r, cc, dtype=torch.float32) for n, l, r, cc in tens},
              str(tmp_path / "f32.safetensors"))
    files = atp.StFiles([str(tmp_path / "f32.safetensors")])
    _expect_einval(lambda: plan.load_weights(files, names, buf.ctypes.data, n_in), "element size")
    files.close()


def test_duplicate_names_across_files(tmp_path):
    c = configs.get(1, w_kind=KIND_TAG16)
    _, paths, _ = _write(c, tmp_path)
    _expect_einval(lambda: atp.StFiles([paths[0], paths[0]]), "appears twice")


def test_truncated_file(tmp_path):
    c = configs.get(1, w_kind=KIND_TAG16)
    _, paths, _ = _write(c, tmp_path)
    raw = open(paths[0], "rb").read()
    p = tmp_path / "cut.safetensors"
    p.write_bytes(raw[:-10])
    _expect_einval(lambda: atp.StFiles([str(p)]), "outside the data")
    p.write_bytes(raw[:5])
    _expect_einval(lambda: atp.StFiles([str(p)]), "shorter than")
    p.write_bytes((1 << 40).to_bytes(8, "little") + b"{}")
    _expect_einval(lambda: atp.StFiles([str(p)]), "does not fit")


@pytest.mark.parametrize("header,match", [
    (b'{"a": {"dtype": "BF16", "shape": [2], "data_offsets": [0, 4]}', "expected"),
    (b'{"a": {"dtype": "BF16", "shape": [2], "data_offsets": [0, 4]}} x', "trailing"),
    (b'{"a": {"dtype": "Q4", "shape": [2], "data_offsets": [0, 4]}}', "unknown dtype"),
    (b'{"a": {"dtype": "BF16", "shape": [3], "data_offsets": [0, 4]}}', "does not match"),
    (b'{"a": {"dtype": "BF16", "shape": [-2], "data_offsets": [0, 4]}}', "non-negative"),
    (b'{"a": {"dtype": "BF16", "shape": [2.5], "data_offsets": [0, 4]}}', "integer"),
    (b'{"a": {"dtype": "BF16", "shape": [2]}}', "lacks"),
    (b'{"a": {"dtype": "BF16", "shape": [2], "data_offsets": [4, 0]}}', "outside"),
    (b'{"a\\x": {"dtype": "BF16", "shape": [2], "data_offsets": [0, 4]}}', "bad escape"),
    (b'{"a": {"dtype": "BF16", "shape": [99999999999999999999], "data_offsets": [0, 4]}}', "overflow"),
])
def test_malformed_headers(tmp_path, header, match):
    p = _raw(tmp_path, header, b"\0" * 4)
    _expect_einval(lambda: atp.StFiles([p]), match)


def test_header_syntax_the_format_allows(tmp_path):
    # escapes, metadata, unknown keys, whitespace, an empty tensor
    meta = {
        "__metadata__": {"format": "pt", "note": "x\"y"},
        "café.\"q\"": {"dtype": "U16", "shape": [2, 2], "data_offsets": [0, 8], "extra": [1, {"z": None}]},
        "empty": {"dtype": "F32", "shape": [0, 5], "data_offsets": [8, 8]},
        "scalar": {"dtype": "I64", "shape": [], "data_offsets": [8, 16]},
    }
    h = json.dumps(meta, indent=2, ensure_ascii=True).encode()
    p = _raw(tmp_path, h, bytes(range(16)))
    files = atp.StFiles([p])
    fi, eb, shape, off, nb = files.find("café.\"q\"")
    assert (fi, eb, shape, off, nb) == (0, 2, (2, 2), 8 + len(h), 8)
    assert files.find("empty")[2:] == ((0, 5), 8 + len(h) + 8, 0)
    assert files.find("scalar")[1:] == (8, (), 8 + len(h) + 8, 8)
    files.close()
