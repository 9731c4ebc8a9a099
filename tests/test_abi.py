"""CPU checks of the C ABI: the library loads and exports every function the header
declares (no compute call is made here)."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xstage.h")
LIB = os.path.join(ROOT, "paper_2607_23264_amd", "libxstage.so")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\*?\s*(xs_\w+)\s*\(", src, flags=re.M)))


def _ensure_built():
    if not os.path.exists(LIB):
        from paper_2607_23264_amd.build import build
        build(verbose=False)


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("xs_route_topk_softmax", "xs_dispatch_layout", "xs_dispatch", "xs_expert_ffn",
                 "xs_combine_send", "xs_combine_reduce", "xs_fused_ep_layer", "xs_gemm_scatter",
                 "xs_model_fit", "xs_model_predict", "xs_xstage_microbench"):
        assert must in names


def test_library_exports_every_declared_symbol():
    _ensure_built()
    lib = ctypes.CDLL(LIB)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    _ensure_built()
    from paper_2607_23264_amd import xstage
    assert sorted(xstage.EXPORTED) == _declared()
