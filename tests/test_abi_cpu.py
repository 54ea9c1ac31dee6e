"""C-ABI checks that need no GPU: the library loads, exports every declared entry point,
and rejects bad arguments synchronously (before any device work)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "surrogate.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(surrogate_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = declared_functions()
    assert len(names) == 27
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTS)


def test_tensor_layout_matches_the_synthetic_generator():
    for w in synth.CONFIGS.values():
        cfg = B.make_config(w.shape)
        specs = synth.tensor_specs(w.shape)
        assert B.surrogate_tensor_count(cfg) == len(specs)
        for i, (name, rows, cols, is_norm) in enumerate(specs):
            r, c, dt = B.surrogate_tensor_shape(cfg, i)
            assert (r, c) == (rows, cols), name
            assert dt == (B.SURR_F32 if is_norm or w.shape.dtype == "f32" else B.SURR_BF16)


@pytest.mark.parametrize("bad", [dict(n_q_heads=5, n_kv_heads=2), dict(head_dim=48),
                                 dict(vocab=1000), dict(d_ff=100), dict(max_pos=0),
                                 dict(n_layers=0)])
def test_unsupported_configs_are_rejected(bad):
    shape = synth.CONFIGS["small"].shape.replace(**bad)
    cfg = B.make_config(shape)
    with pytest.raises(B.SurrogateError) as e:
        B.surrogate_tensor_shape(cfg, 0)
    assert e.value.status in (B.SURR_E_SHAPE,)


def test_load_weights_rejects_wrong_tensor_count_before_allocating():
    cfg = B.make_config(synth.CONFIGS["tiny"].shape)
    ptrs = (ctypes.c_void_p * 3)(1, 1, 1)
    h = ctypes.c_void_p()
    st = B.lib().surrogate_load_weights_tensors(ctypes.byref(cfg), ptrs, 3, 0, None, ctypes.byref(h))
    assert st == B.SURR_E_WEIGHTS and not h.value
    assert b"expected" in B.lib().surrogate_last_error()


def test_select_rejects_bad_arguments_synchronously():
    L = B.lib()
    p = ctypes.c_void_p(16)
    assert L.surrogate_select(p, 0, 0, 0.5, 0, p, p, p, None) == B.SURR_E_INVALID_ARG
    assert L.surrogate_select(p, 65537, 0, 0.5, 0, p, p, p, None) == B.SURR_E_INVALID_ARG
    assert L.surrogate_select(p, 4, 7, 0.5, 0, p, p, p, None) == B.SURR_E_INVALID_ARG
    assert L.surrogate_select(p, 4, 1, 0.5, -1, p, p, p, None) == B.SURR_E_INVALID_ARG
    assert L.surrogate_select(None, 4, 0, 0.5, 0, p, p, p, None) == B.SURR_E_INVALID_ARG


def test_top_score_select_rejects_negative_k():
    L = B.lib()
    p = ctypes.c_void_p(16)
    assert L.surrogate_select(p, 4, 2, 0.0, -1, p, p, p, None) == B.SURR_E_INVALID_ARG


def test_forecast_head_rejects_bad_arguments_synchronously():
    L = B.lib()
    p = ctypes.c_void_p(256)
    m = np.arange(1, 9, dtype=np.float64)
    e = 2.0 ** np.array([-2, -1, -0.5, 0, 0.5, 1, 2])
    md, ed = m.ctypes.data, e.ctypes.data

    def call(n=4, nb=8, m_=md, e_=ed, cut=(1.5,), nc=None, probs=p):
        c = np.asarray(cut, np.float64)
        nc = c.size if nc is None else nc
        return L.surrogate_forecast_head(probs, n, nb, m_, e_, c.ctypes.data if c.size else None,
                                         nc, p, p, None)

    assert call(n=-1) == B.SURR_E_INVALID_ARG
    assert call(nb=0) == B.SURR_E_INVALID_ARG
    assert call(nb=17) == B.SURR_E_INVALID_ARG
    assert call(cut=tuple(range(9)), nc=9) == B.SURR_E_INVALID_ARG
    assert call(m_=None) == B.SURR_E_INVALID_ARG
    assert call(probs=None) == B.SURR_E_INVALID_ARG
    assert call(e_=None) == B.SURR_E_INVALID_ARG
    assert call(cut=(0.2,)) == B.SURR_E_INVALID_ARG       # below the first edge
    assert call(cut=(4.5,)) == B.SURR_E_INVALID_ARG       # above the last edge
    assert call(cut=(float("nan"),)) == B.SURR_E_INVALID_ARG
    bad_e = e.copy()
    bad_e[3] = bad_e[2]
    assert call(e_=bad_e.ctypes.data) == B.SURR_E_INVALID_ARG
    bad_m = m.copy()
    bad_m[5] = np.inf
    assert call(m_=bad_m.ctypes.data) == B.SURR_E_INVALID_ARG
    assert call(nb=1, cut=(1.0,)) == B.SURR_E_INVALID_ARG
    assert b"cutoff" in L.surrogate_last_error() or L.surrogate_last_error()


def test_prefix_calls_reject_bad_arguments_synchronously():
    L = B.lib()
    p = ctypes.c_void_p(256)
    lens = np.array([3], np.int32)
    pid = np.array([0], np.int32)
    vid = np.array([1], np.int32)
    h = ctypes.c_void_p()
    assert L.surrogate_prefix_build(None, p, 4, lens.ctypes.data, 1, p, 1 << 20, None,
                                    ctypes.byref(h)) == B.SURR_E_INVALID_ARG and not h.value
    assert L.surrogate_score_suffixes(None, p, pid.ctypes.data, p, 4, lens.ctypes.data, 1,
                                      vid.ctypes.data, 1, p, 1 << 20, p, None, p, None,
                                      None) == B.SURR_E_INVALID_ARG
    n = ctypes.c_size_t()
    assert L.surrogate_prefix_cache_bytes(None, ctypes.byref(n)) == B.SURR_E_INVALID_ARG
    L.surrogate_prefix_free(None)  # ignored


def test_evaluate_rejects_bad_arguments_synchronously():
    L = B.lib()
    p = ctypes.c_void_p(256)
    m = np.arange(1, 9, dtype=np.float64)
    e = 2.0 ** np.array([-2, -1, -0.5, 0, 0.5, 1, 2])
    c = np.array([0.25], np.float64)
    sz = ctypes.c_size_t()
    assert L.surrogate_evaluate_workspace_size(0, 1, ctypes.byref(sz)) == B.SURR_E_INVALID_ARG
    assert L.surrogate_evaluate_workspace_size(65537, 1, ctypes.byref(sz)) == B.SURR_E_INVALID_ARG
    assert L.surrogate_evaluate_workspace_size(10, 9, ctypes.byref(sz)) == B.SURR_E_INVALID_ARG
    assert L.surrogate_evaluate_workspace_size(10, 5, ctypes.byref(sz)) == B.SURR_OK and sz.value

    def call(n=10, nb=8, m_=m, e_=e, c_=c, ws_bytes=1 << 20):
        return L.surrogate_evaluate(p, p, n, nb, m_.ctypes.data, e_.ctypes.data, c_.ctypes.data,
                                    c_.size, p, ws_bytes, None, None, None, p, None)

    assert call(nb=1) == B.SURR_E_INVALID_ARG
    assert call(nb=17) == B.SURR_E_INVALID_ARG
    assert call(ws_bytes=16) == B.SURR_E_WORKSPACE
    assert call(c_=np.array([0.0])) == B.SURR_E_INVALID_ARG
    assert call(c_=np.array([1.5])) == B.SURR_E_INVALID_ARG
    bad = e.copy()
    bad[2] = -1.0
    assert call(e_=bad) == B.SURR_E_INVALID_ARG
    assert L.surrogate_evaluate(None, p, 10, 8, m.ctypes.data, e.ctypes.data, c.ctypes.data, 1, p,
                                1 << 20, None, None, None, p, None) == B.SURR_E_INVALID_ARG

    # the variant on the fixed scratch checks the same arguments before any device call
    def call_na(n=10, nb=8, m_=m, e_=e, c_=c, probs=p):
        return L.surrogate_evaluate_noalloc(probs, p, n, nb, m_.ctypes.data, e_.ctypes.data,
                                            c_.ctypes.data, c_.size, None, None, None, p, None)

    assert call_na(nb=1) == B.SURR_E_INVALID_ARG
    assert call_na(n=65537) == B.SURR_E_INVALID_ARG  # past the scratch's maximum call
    assert call_na(n=0) == B.SURR_E_INVALID_ARG
    assert call_na(c_=np.zeros(9) + 0.5) == B.SURR_E_INVALID_ARG
    assert call_na(c_=np.array([1.5])) == B.SURR_E_INVALID_ARG
    assert call_na(e_=bad) == B.SURR_E_INVALID_ARG
    assert call_na(probs=None) == B.SURR_E_INVALID_ARG


def test_cache_calls_reject_bad_arguments_synchronously():
    L = B.lib()
    p = ctypes.c_void_p(256)
    cap = np.array([64], np.int32)
    h = ctypes.c_void_p()
    assert L.surrogate_cache_create(None, 1, cap.ctypes.data, ctypes.byref(h)) == B.SURR_E_INVALID_ARG
    lens = np.array([1], np.int32)
    assert L.surrogate_cache_extend(None, p, lens.ctypes.data, p, 1, lens.ctypes.data, 1, None, p,
                                    1 << 20, None, None, None) == B.SURR_E_INVALID_ARG
    assert L.surrogate_cache_lengths(None, lens.ctypes.data) == B.SURR_E_INVALID_ARG
    assert L.surrogate_cache_reset(None, lens.ctypes.data, 1) == B.SURR_E_INVALID_ARG


def test_score_pairs_rejects_null_model():
    L = B.lib()
    p = ctypes.c_void_p(256)
    lens = np.array([3], np.int32)
    vid = np.array([1], np.int32)
    st = L.surrogate_score_pairs(None, p, 4, lens.ctypes.data, 1, vid.ctypes.data, 1, p, 1 << 20,
                                 p, None, p, None, None)
    assert st == B.SURR_E_INVALID_ARG


def test_status_strings():
    L = B.lib()
    for s in range(0, -9, -1):
        assert L.surrogate_status_string(s)
    assert L.surrogate_status_string(-3) == b"token id out of range"


def test_library_has_no_unresolved_kernel_stubs():
    # a kernel template dropped by the host compilation pass leaves an undefined launch
    # stub that only fails when that kernel is first launched
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    assert "__device_stub__" not in out


# ---------------------------------------------------------------- weight files
def _config_tuple(cfg):
    return tuple(getattr(cfg, f) for f, _ in B.surrogate_config._fields_)


@pytest.mark.parametrize("name,layers", [("tiny", 2), ("small", 1), ("7b", 1)])
def test_weight_file_round_trip_config(tmp_path, name, layers):
    """synth.write_weight_file writes the format the library reads: the declared
    configuration comes back field for field, the tensor bytes sit where the header says."""
    shape = synth.CONFIGS[name].shape.replace(n_layers=layers)
    if name == "7b":  # full width, a tiny vocabulary keeps the file small
        shape = shape.replace(vocab=256)
    W = synth.make_weights(shape, gain_std=0.1)
    path = tmp_path / "w.surw"
    synth.write_weight_file(path, shape, W)
    got = B.surrogate_weight_file_config(str(path))
    assert _config_tuple(got) == _config_tuple(B.make_config(shape))
    raw = path.read_bytes()
    assert raw[:8] == b"SURRWGT1"
    hl = int.from_bytes(raw[8:16], "little")
    import json
    head = json.loads(raw[16:16 + hl])
    for (n, dt, shp, a), t in zip(synth.file_tensors(shape, W), head["tensors"]):
        assert t["name"] == n and t["offset"] % 4096 == 0
        a = np.ascontiguousarray(a)
        assert raw[t["offset"]: t["offset"] + a.nbytes] == a.tobytes(), n


def _mutations(raw):
    """Malformed variants of a valid file, each with what is wrong."""
    import json
    hl = int.from_bytes(raw[8:16], "little")
    head = json.loads(raw[16:16 + hl])
    first = head["tensors"][0]["offset"]

    def with_header(h):  # the blobs stay where the original offsets put them
        hb = json.dumps(h).encode()
        out = raw[:8] + len(hb).to_bytes(8, "little") + hb
        return out + bytes(first - len(out)) + raw[first:] if len(out) <= first else None

    def edit(fn):
        h = json.loads(json.dumps(head))
        fn(h)
        return with_header(h)

    yield "bad magic", b"XURRWGT1" + raw[8:]
    yield "truncated preamble", raw[:10]
    yield "header length past the end", raw[:8] + (len(raw)).to_bytes(8, "little") + raw[16:]
    yield "header length zero", raw[:8] + (0).to_bytes(8, "little") + raw[16:]
    yield "truncated last tensor", raw[:-100]
    yield "broken JSON", raw[:16 + hl // 2] + b"}" + raw[16 + hl // 2 + 1:]
    yield "wrong format", edit(lambda h: h.update(format="other"))
    yield "wrong version", edit(lambda h: h.update(version=2))
    yield "missing config field", edit(lambda h: h["config"].pop("d_ff"))
    yield "extra config field", edit(lambda h: h["config"].update(extra=1))
    yield "bad dtype", edit(lambda h: h["config"].update(dtype="f16"))
    yield "unsupported shape", edit(lambda h: h["config"].update(head_dim=48))
    yield "fractional size", edit(lambda h: h["config"].update(d_model=128.5))
    yield "tensor missing", edit(lambda h: h["tensors"].pop())
    yield "tensors swapped", edit(lambda h: h["tensors"].__setitem__(
        slice(1, 3), [h["tensors"][2], h["tensors"][1]]))
    yield "wrong tensor dtype", edit(lambda h: h["tensors"][1].update(dtype="bf16"))
    yield "wrong shape", edit(lambda h: h["tensors"][2].update(
        shape=[h["tensors"][2]["shape"][0] + 1, h["tensors"][2]["shape"][1]]))
    yield "misaligned offset", edit(lambda h: h["tensors"][3].update(offset=h["tensors"][3]["offset"] + 8))
    yield "overlapping tensors", edit(lambda h: h["tensors"][3].update(offset=h["tensors"][2]["offset"]))
    yield "negative offset", edit(lambda h: h["tensors"][0].update(offset=-4096))
    yield "offset past the end", edit(lambda h: h["tensors"][-1].update(offset=1 << 40))
    yield "extra tensor key", edit(lambda h: h["tensors"][0].update(extra=0))


def test_malformed_weight_files_are_rejected_before_device_work(tmp_path):
    shape = synth.CONFIGS["tiny"].shape
    W = synth.make_weights(shape)
    good = tmp_path / "good.surw"
    synth.write_weight_file(good, shape, W)
    raw = good.read_bytes()
    L = B.lib()
    cfg = B.surrogate_config()
    h = ctypes.c_void_p()
    seen = 0
    for what, data in _mutations(raw):
        if data is None:
            continue
        p = tmp_path / "bad.surw"
        p.write_bytes(data)
        assert L.surrogate_weight_file_config(str(p).encode(), ctypes.byref(cfg)) == B.SURR_E_WEIGHTS, what
        # the loader checks the same header before it touches a device
        assert L.surrogate_load_weights(str(p).encode(), None, ctypes.byref(h)) == B.SURR_E_WEIGHTS, what
        assert not h.value
        seen += 1
    assert seen >= 20
    assert L.surrogate_weight_file_config(str(tmp_path / "none.surw").encode(),
                                          ctypes.byref(cfg)) == B.SURR_E_IO
    assert L.surrogate_weight_file_config(str(tmp_path).encode(), ctypes.byref(cfg)) == B.SURR_E_IO
    assert L.surrogate_weight_file_config(None, ctypes.byref(cfg)) == B.SURR_E_INVALID_ARG
    assert L.surrogate_load_weights(None, None, ctypes.byref(h)) == B.SURR_E_INVALID_ARG
