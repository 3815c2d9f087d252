"""The C ABI on the CPU: the library loads, exports what include/ace.h
declares, and rejects invalid calls on the host before any launch (no GPU is
touched by these tests).  The product path has no CPU or oracle fallback."""
import ctypes
import os
import re

import pytest

import paper_2609_05228_amd as ace
from paper_2609_05228_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ace.h")
FAKE = 0x10000  # aligned, never dereferenced: every call below returns before any launch


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ace_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = ace.lib()
    names = header_functions()
    assert {"ace_moe_forward", "ace_moe_workspace_size", "ace_status_string", "ace_abi_version"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in ace.h but not exported"


def test_version_and_status_strings():
    m = re.search(r"#define ACE_ABI_VERSION (\d+)", open(HEADER).read())
    assert ace.abi_version() == int(m.group(1))
    for code, word in [(0, "ACE_OK"), (-1, "INVALID_ARG"), (-2, "UNSUPPORTED"), (-3, "WORKSPACE"), (-4, "HIP"),
                       (-5, "SCRATCH_LIMIT")]:
        assert word in ace.status_string(code)
    assert "unknown" in ace.status_string(12345)


def _desc(**kw):
    base = dict(T=64, d=256, N=8, k=2, m=512, dtype=_lib.ACE_BF16, tau=0.1)
    base.update(kw)
    return ace.make_desc(base.pop("T"), base.pop("d"), base.pop("N"), base.pop("k"), base.pop("m"),
                         base.pop("dtype"), base.pop("tau"), **base)


def _call(desc, x=FAKE, w=None, o=None, ws=0, ws_bytes=0):
    if w is None:
        w = _lib.Weights(*([FAKE] * 3 + [FAKE] * 3 + [0, 0, 0] + [FAKE, FAKE]))
        w.b_router = 0
    if o is None:
        o = _lib.Outputs(FAKE, FAKE, FAKE, 0, 0, 0, 0, 0)
    return ace.forward_raw(desc, x, w, o, ws, ws_bytes, 0)


def test_workspace_size():
    assert ace.workspace_size(_desc()) > 0
    assert ace.workspace_size(_desc(T=0)) == 0
    big = ace.workspace_size(_desc(T=4096, d=2048, N=128, k=8, m=768))
    assert big > 4096 * 2048 * 2 + 4096 * 8 * (768 + 2048) * 2  # x_in, H and Y at least
    # past the small-batch path (fp32 split-K partials), fp32 buffers are the larger ones
    assert ace.workspace_size(_desc(T=256, dtype=_lib.ACE_F32)) > ace.workspace_size(_desc(T=256))


@pytest.mark.parametrize("kw,status", [
    (dict(k=9, N=8), _lib.ACE_ERR_INVALID_ARG),            # k > N
    (dict(m_min=0), _lib.ACE_ERR_INVALID_ARG),
    (dict(m_min=3), _lib.ACE_ERR_INVALID_ARG),             # m_min > k
    (dict(dtype=7), _lib.ACE_ERR_INVALID_ARG),
    (dict(tau=float("nan")), _lib.ACE_ERR_INVALID_ARG),
    (dict(eps=-1.0), _lib.ACE_ERR_INVALID_ARG),
    (dict(T=-1), _lib.ACE_ERR_INVALID_ARG),
    (dict(N=300, k=2), _lib.ACE_ERR_UNSUPPORTED),
    (dict(N=16, k=9), _lib.ACE_ERR_UNSUPPORTED),
    (dict(d=200), _lib.ACE_ERR_UNSUPPORTED),
    (dict(m=100), _lib.ACE_ERR_UNSUPPORTED),
    (dict(n_shared=1, m_shared=96), _lib.ACE_ERR_UNSUPPORTED),
])
def test_invalid_descriptors(kw, status):
    assert _call(_desc(**kw)) == status


def test_null_and_misaligned_pointers():
    d = _desc()
    assert _call(d, x=0) == _lib.ACE_ERR_INVALID_ARG
    assert _call(d, x=FAKE + 2) == _lib.ACE_ERR_INVALID_ARG
    w = _lib.Weights(FAKE, FAKE, 0, FAKE, FAKE, 0, 0, 0, 0, FAKE, FAKE)  # w_down missing
    assert _call(d, w=w) == _lib.ACE_ERR_INVALID_ARG
    o = _lib.Outputs(FAKE, 0, FAKE, 0, 0, 0, 0, 0)                         # topk_idx missing
    assert _call(d, o=o) == _lib.ACE_ERR_INVALID_ARG
    # shared expert requested without its weights
    assert _call(_desc(n_shared=1, m_shared=128)) == _lib.ACE_ERR_INVALID_ARG
    # scores requested without a scores buffer
    assert _call(_desc(write_scores=True)) == _lib.ACE_ERR_INVALID_ARG
    # unknown flag bit, and fusion rules past ACE_FUSION_SCORE
    for flags in (1 << 7, 6 << _lib.ACE_FUSION_SHIFT, 7 << _lib.ACE_FUSION_SHIFT):
        d2 = _desc()
        d2.flags = flags
        assert _call(d2) == _lib.ACE_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        _desc(fusion="median")


def test_workspace_checked_before_launch():
    d = _desc()
    need = ace.workspace_size(d)
    assert _call(d, ws=0, ws_bytes=need) == _lib.ACE_ERR_WORKSPACE
    assert _call(d, ws=FAKE, ws_bytes=need - 1) == _lib.ACE_ERR_WORKSPACE
    assert _call(d, ws=FAKE + 16, ws_bytes=need) == _lib.ACE_ERR_WORKSPACE  # not 256-byte aligned


def test_empty_batch_is_a_no_op():
    assert _call(_desc(T=0), x=0, o=_lib.Outputs()) == _lib.ACE_OK


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libace.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        _lib.lib()


def test_product_path_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2609_05228_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\boracle\b", text), f"{f} mentions the oracle"


def test_tau_map_validation():
    need = ace.tau_workspace_size()
    assert need > 0
    ok = dict(scores=FAKE, n_rows=4, k=8, m_min=1, qs=[0.5], tau=FAKE, ws=FAKE, ws_bytes=need)

    def call(**kw):
        a = dict(ok, **kw)
        return ace.tau_map_raw(a["scores"], a["n_rows"], a["k"], a["m_min"], a["qs"], a["tau"], 0, 0,
                               a["ws"], a["ws_bytes"], 0)
    for kw in (dict(k=0), dict(k=9), dict(m_min=0), dict(m_min=9, k=8), dict(n_rows=-1), dict(qs=[]),
               dict(qs=[0.5] * 9), dict(qs=[1.01]), dict(qs=[-1e-9]), dict(qs=[float("nan")]),
               dict(tau=0), dict(scores=0), dict(scores=FAKE + 2)):
        assert call(**kw) == _lib.ACE_ERR_INVALID_ARG, kw
    for kw in (dict(ws=0), dict(ws_bytes=need - 1), dict(ws=FAKE + 16)):
        assert call(**kw) == _lib.ACE_ERR_WORKSPACE, kw


def test_build_tables_validation():
    d = _desc(d=256, N=8, m=512)
    need = ace.tables_workspace_size(d)
    assert need > 0

    def call(desc=d, w=None, gsp=FAKE, rcr=FAKE, ws=FAKE, ws_bytes=need):
        if w is None:
            w = _lib.Weights(FAKE, FAKE, 0, FAKE, FAKE, FAKE, 0, 0, 0, 0, 0)
        return ace.build_tables_raw(desc, w, gsp, rcr, 0, 0, ws, ws_bytes, 0)
    assert call(desc=_desc(m=96)) == _lib.ACE_ERR_UNSUPPORTED       # m % 64
    assert call(desc=_desc(d=200, m=512)) == _lib.ACE_ERR_UNSUPPORTED
    assert call(gsp=0) == _lib.ACE_ERR_INVALID_ARG
    assert call(w=_lib.Weights(FAKE, FAKE, 0, FAKE, 0, FAKE, 0, 0, 0, 0, 0)) == _lib.ACE_ERR_INVALID_ARG
    assert call(w=_lib.Weights(FAKE + 8, FAKE, 0, FAKE, FAKE, FAKE, 0, 0, 0, 0, 0)) == _lib.ACE_ERR_INVALID_ARG
    assert call(ws=0) == _lib.ACE_ERR_WORKSPACE
    assert call(ws_bytes=need - 1) == _lib.ACE_ERR_WORKSPACE

def test_noalloc_validates_and_refuses_oversized_layers_on_the_host():
    """The no-allocation entry point checks its arguments like ace_moe_forward and
    refuses a layer whose workspace exceeds its static scratch before touching any
    device (these calls return without a GPU)."""
    w = _lib.Weights(*([FAKE] * 3 + [FAKE] * 3 + [0, 0, 0] + [FAKE, FAKE]))
    w.b_router = 0
    o = _lib.Outputs(FAKE, FAKE, FAKE, 0, 0, 0, 0, 0)
    big = _desc(T=4096, d=2048, N=128, k=8, m=768)
    m = re.search(r"#define ACE_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == _lib.NOALLOC_SCRATCH_BYTES
    assert ace.workspace_size(big) > _lib.NOALLOC_SCRATCH_BYTES
    assert _lib.forward_noalloc_raw(big, FAKE, w, o, 0) == _lib.ACE_ERR_SCRATCH_LIMIT
    edge = _desc(T=1362, d=2048, N=128, k=8, m=768)
    assert ace.workspace_size(edge) > _lib.NOALLOC_SCRATCH_BYTES
    assert _lib.forward_noalloc_raw(edge, FAKE, w, o, 0) == _lib.ACE_ERR_SCRATCH_LIMIT
    assert ace.workspace_size(_desc(T=1361, d=2048, N=128, k=8, m=768)) <= _lib.NOALLOC_SCRATCH_BYTES
    assert _lib.forward_noalloc_raw(_desc(k=9, N=8), FAKE, w, o, 0) == _lib.ACE_ERR_INVALID_ARG
    assert _lib.forward_noalloc_raw(_desc(d=200), FAKE, w, o, 0) == _lib.ACE_ERR_UNSUPPORTED
    assert _lib.forward_noalloc_raw(_desc(T=0), FAKE, w, o, 0) == _lib.ACE_OK
    o0 = _lib.Outputs(0, FAKE, FAKE, 0, 0, 0, 0, 0)
    assert _lib.forward_noalloc_raw(_desc(), FAKE, w, o0, 0) == _lib.ACE_ERR_INVALID_ARG
