"""The C-ABI library on the host: it loads, exports every declared entry
point, and its argument checks reject bad calls before touching the GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "uattn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(uattn_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_35140_amd import uattn
    if not os.path.exists(uattn.LIB_PATH):
        from paper_2609_35140_amd import build
        build.build()
    return uattn.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["uattn_prefill", "uattn_decode", "uattn_decode_workspace_bytes", "uattn_logprob", "uattn_kv_write",
              "uattn_status_string", "uattn_abi_version"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n
    # no C++ mangling on the boundary
    so = ctypes.CDLL(os.path.join(ROOT, "paper_2609_35140_amd", "libuattn.so"))
    for n in declared_functions():
        getattr(so, n)


def test_abi_version_and_status_strings(lib):
    from paper_2609_35140_amd import uattn
    assert uattn.abi_version() == 1
    assert uattn.status_string(0) == "UATTN_OK"
    for code in range(1, 6):
        assert uattn.status_string(code).startswith("UATTN_E")
    assert "UNKNOWN" in uattn.status_string(99)


def _r256(x):
    return (x + 255) // 256 * 256


def test_workspace_bytes(lib):
    from paper_2609_35140_amd import uattn
    assert uattn.decode_workspace_bytes(8, 256, 32, 128) == 0        # one chunk: no partials
    # counters [B*Hq int32] + acc [B*Hq*nchunk*d fp32] + (m, l) [B*Hq*nchunk*2 fp32], each 256-aligned
    assert uattn.decode_workspace_bytes(8, 257, 32, 128) == _r256(8 * 32 * 4) + 8 * 32 * 2 * 128 * 4 + _r256(8 * 32 * 2 * 2 * 4)
    assert uattn.decode_workspace_bytes(8, 4096, 32, 128) == _r256(8 * 32 * 4) + 8 * 32 * 16 * 128 * 4 + _r256(8 * 32 * 16 * 2 * 4)
    assert uattn.decode_workspace_bytes(3, 300, 5, 64) == _r256(3 * 5 * 4) + _r256(3 * 5 * 2 * 64 * 4) + _r256(3 * 5 * 2 * 2 * 4)
    # chunk slots rounded up to even: 3 chunks take 4 slots
    assert uattn.decode_workspace_bytes(2, 600, 8, 128) == _r256(2 * 8 * 4) + 2 * 8 * 4 * 128 * 4 + _r256(2 * 8 * 4 * 2 * 4)
    assert uattn.decode_workspace_bytes(0, 4096, 32, 128) == 0
    assert uattn.decode_workspace_bytes(1, -5, 32, 128) == 0


P = ctypes.c_void_p


def _prefill(lib, **kw):
    a = dict(q=P(16), k=P(16), v=P(16), cu=P(16), ns=1, T=4, maxs=4, hq=4, hkv=2, d=128, scale=0.1,
             out=P(32), lse=None, stream=None)
    a.update(kw)
    return lib.uattn_prefill(a["q"], a["k"], a["v"], a["cu"], a["ns"], a["T"], a["maxs"], a["hq"], a["hkv"], a["d"],
                             a["scale"], a["out"], a["lse"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(hq=3, hkv=2), 1), (dict(hkv=0), 1), (dict(ns=-1), 1), (dict(scale=0.0), 1),
    (dict(scale=float("inf")), 1), (dict(scale=float("nan")), 1), (dict(scale=-1.0), 1),
    (dict(d=96), 2), (dict(d=256), 2), (dict(q=None), 1), (dict(out=None), 1), (dict(q=P(18)), 1),
    (dict(ns=0), 0), (dict(T=0), 0), (dict(maxs=0), 0),
])
def test_prefill_argument_checks(lib, kw, code):
    assert _prefill(lib, **kw) == code


def _decode(lib, **kw):
    a = dict(q=P(16), kp=P(16), vp=P(16), bt=P(16), sl=P(16), B=2, maxp=4, page=16, npages=10, maxs=64, hq=8, hkv=2, d=128,
             scale=0.1, out=P(32), lse=None, ws=None, wsb=0, stream=None)
    a.update(kw)
    return lib.uattn_decode(a["q"], a["kp"], a["vp"], a["bt"], a["sl"], a["B"], a["maxp"], a["page"], a["npages"], a["maxs"],
                            a["hq"], a["hkv"], a["d"], a["scale"], a["out"], a["lse"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(hq=9), 1), (dict(page=24), 2), (dict(page=8), 2), (dict(d=80), 2), (dict(hq=66, hkv=2), 2),
    (dict(maxp=3), 1), (dict(maxs=0), 1), (dict(bt=None), 1), (dict(scale=0.0), 1),
    (dict(npages=0), 1), (dict(npages=-1), 1), (dict(maxs=(1 << 24) + 1, maxp=1 << 20), 2), (dict(maxs=300, maxp=19), 3), (dict(maxs=300, maxp=19, ws=P(64), wsb=100), 3), (dict(B=0), 0),
])
def test_decode_argument_checks(lib, kw, code):
    assert _decode(lib, **kw) == code


@pytest.mark.parametrize("args,code", [
    ((P(16), 8, P(16), 4, 0, 1.0, P(16), None), 1),       # vocab 0
    ((P(16), 4, P(16), 4, 8, 1.0, P(16), None), 1),       # stride < vocab
    ((P(16), 12, P(16), 4, 8, 1.0, P(16), None), 1),      # stride not a multiple of 8
    ((P(18), 8, P(16), 4, 8, 1.0, P(16), None), 1),       # misaligned logits
    ((P(16), 8, P(16), 4, 8, 0.0, P(16), None), 1),       # temperature
    ((P(16), 8, P(16), 0, 8, 1.0, P(16), None), 0),       # no rows
])
def test_logprob_argument_checks(lib, args, code):
    assert lib.uattn_logprob(*args) == code


def _kv_write(lib, **kw):
    a = dict(kn=P(16), vn=P(16), stride=256, bt=P(16), si=P(16), pos=P(16), N=4, B=2, maxp=4, page=16, npages=10,
             hkv=2, d=128, kp=P(16), vp=P(16), stream=None)
    a.update(kw)
    return lib.uattn_kv_write(a["kn"], a["vn"], a["stride"], a["bt"], a["si"], a["pos"], a["N"], a["B"], a["maxp"],
                              a["page"], a["npages"], a["hkv"], a["d"], a["kp"], a["vp"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(d=96), 2), (dict(page=24), 2), (dict(page=8), 2), (dict(stride=200), 1), (dict(stride=260), 1),
    (dict(hkv=0), 1), (dict(N=-1), 1), (dict(kn=None), 1), (dict(vp=None), 1), (dict(pos=None), 1),
    (dict(kn=P(18)), 1), (dict(kp=P(24)), 1), (dict(N=0), 0), (dict(npages=0), 0), (dict(B=0), 0),
])
def test_kv_write_argument_checks(lib, kw, code):
    assert _kv_write(lib, **kw) == code


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2609_35140_amd import uattn
    monkeypatch.setattr(uattn, "_lib", None)
    monkeypatch.setattr(uattn, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(uattn.UattnError):
        uattn.abi_version()


@pytest.mark.parametrize("kw,code", [
    (dict(d=96), 2), (dict(eps=-1.0), 1), (dict(eps=float("nan")), 1), (dict(maxpos=0), 1), (dict(hq=0), 1),
    (dict(q=None), 1), (dict(cs=None), 1), (dict(cs=P(20)), 1), (dict(T=-1), 1), (dict(T=0), 0),
])
def test_qk_norm_rope_argument_checks(lib, kw, code):
    a = dict(q=P(16), k=P(16), pos=P(16), qw=P(16), kw=P(16), eps=1e-6, cs=P(16), maxpos=10, T=4, hq=4, hkv=2, d=128,
             qo=P(16), ko=P(16), stream=None)
    a.update(kw)
    assert lib.uattn_qk_norm_rope(a["q"], a["k"], a["pos"], a["qw"], a["kw"], a["eps"], a["cs"], a["maxpos"], a["T"],
                                  a["hq"], a["hkv"], a["d"], a["qo"], a["ko"], a["stream"]) == code


@pytest.mark.parametrize("args,code", [
    ((P(16), 10, 96, 1e4, None), 2), ((P(16), 10, 128, 1.0, None), 1), ((P(16), -1, 128, 1e4, None), 1),
    ((None, 10, 128, 1e4, None), 1), ((P(16), 0, 128, 1e4, None), 0),
])
def test_rope_cache_argument_checks(lib, args, code):
    assert lib.uattn_rope_cache(*args) == code


@pytest.mark.parametrize("kw,code", [
    (dict(H=100), 1), (dict(H=0), 1), (dict(hs=512), 1), (dict(ws=1020), 1), (dict(os=1004), 1), (dict(os=999), 1),
    (dict(h=P(18)), 1), (dict(o=None), 1), (dict(T=-1), 1), (dict(T=0), 0), (dict(V=0), 0),
])
def test_lm_head_argument_checks(lib, kw, code):
    a = dict(h=P(16), hs=1024, w=P(16), ws=1024, T=4, V=1000, H=1024, o=P(16), os=1000, stream=None)
    a.update(kw)
    assert lib.uattn_lm_head(a["h"], a["hs"], a["w"], a["ws"], a["T"], a["V"], a["H"], a["o"], a["os"], a["stream"]) == code


def test_backward_workspace_bytes(lib):
    from paper_2609_35140_amd import uattn
    assert uattn.prefill_backward_workspace_bytes(1000, 32) == 2 * 1000 * 32 * 4   # D and lse*log2(e) per row
    assert uattn.prefill_backward_workspace_bytes(0, 32) == 0
    assert uattn.prefill_backward_workspace_bytes(5, -1) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(hq=3, hkv=2), 1), (dict(hkv=0), 1), (dict(ns=-1), 1), (dict(scale=0.0), 1), (dict(scale=float("nan")), 1),
    (dict(d=96), 2), (dict(q=None), 1), (dict(out=None), 1), (dict(dout=None), 1), (dict(lse=None), 1),
    (dict(dq=None), 1), (dict(dk=None), 1), (dict(dv=None), 1), (dict(dout=P(40)), 1), (dict(lse=P(18)), 1),
    (dict(ws=None), 3), (dict(wsb=127), 3), (dict(ws=P(1032)), 3),
    (dict(ns=0), 0), (dict(T=0), 0), (dict(maxs=0), 0),
])
def test_backward_argument_checks(lib, kw, code):
    a = dict(q=P(16), k=P(16), v=P(16), out=P(16), dout=P(16), lse=P(16), cu=P(16), ns=1, T=4, maxs=4, hq=4, hkv=2,
             d=128, scale=0.1, dq=P(16), dk=P(16), dv=P(16), ws=P(1024), wsb=128, stream=None)
    a.update(kw)
    assert lib.uattn_prefill_backward(a["q"], a["k"], a["v"], a["out"], a["dout"], a["lse"], a["cu"], a["ns"], a["T"],
                                      a["maxs"], a["hq"], a["hkv"], a["d"], a["scale"], a["dq"], a["dk"], a["dv"],
                                      a["ws"], a["wsb"], a["stream"]) == code


def test_decode_noalloc_limits(lib):
    from paper_2609_35140_amd import uattn
    assert uattn.decode_scratch_limit() == 64 << 20
    # sizes the static scratch holds: the Qwen-style and long-context decode batches
    assert uattn.decode_workspace_bytes(8, 4096, 32, 128) <= uattn.decode_scratch_limit()
    assert uattn.decode_workspace_bytes(8, 32768, 64, 128) <= uattn.decode_scratch_limit()
    # ... and one it does not: 512 sequences of 16K keys
    assert uattn.decode_workspace_bytes(512, 16384, 32, 128) > uattn.decode_scratch_limit()


def _decode_noalloc(lib, **kw):
    a = dict(q=P(16), kp=P(16), vp=P(16), bt=P(16), sl=P(16), B=2, maxp=4, page=16, npages=10, maxs=64, hq=8, hkv=2,
             d=128, scale=0.1, out=P(32), lse=None, stream=None)
    a.update(kw)
    return lib.uattn_decode_noalloc(a["q"], a["kp"], a["vp"], a["bt"], a["sl"], a["B"], a["maxp"], a["page"],
                                    a["npages"], a["maxs"], a["hq"], a["hkv"], a["d"], a["scale"], a["out"], a["lse"],
                                    a["stream"])


# single-chunk sizes (no scratch needed, so no HIP call before the checks) and
# sizes beyond the static array (refused by host arithmetic alone)
@pytest.mark.parametrize("kw,code", [
    (dict(hq=9), 1), (dict(page=24), 2), (dict(d=80), 2), (dict(maxp=3), 1), (dict(maxs=0), 1), (dict(bt=None), 1),
    (dict(scale=0.0), 1), (dict(B=0), 0),
    (dict(B=512, maxs=16384, maxp=1024, hq=32, hkv=8), 5), (dict(B=64, maxs=65536, maxp=4096, hq=64, hkv=8), 5),
])
def test_decode_noalloc_argument_checks(lib, kw, code):
    assert _decode_noalloc(lib, **kw) == code


def test_ceilings_library_exports_its_header():
    from paper_2609_35140_amd import build, ceilings
    if not os.path.exists(ceilings.LIB_PATH):
        build.build()
    src = open(os.path.join(ROOT, "include", "uattn_ceilings.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(uattn_[a-z_0-9]+)\s*\(", src)))
    assert names == ["uattn_ceiling_mfma", "uattn_ceiling_read", "uattn_ceiling_read_grid"]
    so = ctypes.CDLL(ceilings.LIB_PATH)
    for n in names:
        getattr(so, n)
    lib = ceilings.lib()
    # argument checks before any GPU call
    assert lib.uattn_ceiling_read(P(16), None, 4, 4096, 0, P(16), None) == 1      # block not a multiple of 16 KB
    assert lib.uattn_ceiling_read(P(18), None, 4, 16384, 0, P(16), None) == 1     # misaligned
    assert lib.uattn_ceiling_read(P(16), None, 4, 16384, 2, P(16), None) == 1     # unknown flag
    assert lib.uattn_ceiling_read(P(16), None, 0, 16384, 1, P(16), None) == 0     # nothing to read
    assert lib.uattn_ceiling_mfma(0, 10, P(16), None) == 1


def test_lm_head_logprob_workspace_and_argument_checks(lib):
    from paper_2609_35140_amd import uattn
    # two fp32 partials per (row, 256-entry vocab tile) plus the target logit per row
    assert uattn.lm_head_logprob_workspace_bytes(8192, 151936) == (2 * 594 + 1) * 8192 * 4
    assert uattn.lm_head_logprob_workspace_bytes(3, 256) == 3 * 3 * 4
    assert uattn.lm_head_logprob_workspace_bytes(0, 100) == 0

    def call(**kw):
        a = dict(h=P(16), hs=1024, w=P(16), ws=1024, tg=P(16), T=4, V=1000, H=1024, it=1.0, lp=P(16), lg=None,
                 ls=0, wk=P(16), wkb=1 << 20, stream=None)
        a.update(kw)
        return lib.uattn_lm_head_logprob(a["h"], a["hs"], a["w"], a["ws"], a["tg"], a["T"], a["V"], a["H"], a["it"],
                                         a["lp"], a["lg"], a["ls"], a["wk"], a["wkb"], a["stream"])
    for kw, code in [(dict(H=100), 1), (dict(hs=512), 1), (dict(it=0.0), 1), (dict(it=float("nan")), 1),
                     (dict(tg=None), 1), (dict(lp=None), 1), (dict(h=P(18)), 1), (dict(V=0), 1),
                     (dict(lg=P(16), ls=999), 1), (dict(lg=P(18), ls=1000), 1), (dict(wk=None), 3), (dict(wkb=100), 3),
                     (dict(wk=P(18)), 3), (dict(T=0), 0), (dict(T=-1), 1)]:
        assert call(**kw) == code, kw
