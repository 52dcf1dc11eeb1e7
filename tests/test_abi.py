"""The C ABI: library loads, exports every symbol include/lsgd.h declares,
and the host-only calls validate their arguments. No GPU work is launched."""
import ctypes
import os
import re

import pytest

import workloads as wk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lsgd.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lsgd_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("lsgd_init_replicas", "lsgd_local_step", "lsgd_average",
                 "lsgd_run_round"):
        assert must in names


def test_library_exports_every_declared_symbol():
    from paper_1808_07217_amd import lsgd as L
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(_declared()) == set(L.EXPORTED)


@pytest.mark.parametrize("name", [n for n, w in wk.WORKLOADS.items()
                                  if w.model == "mlp"])
def test_param_count_matches_layout(name):
    from paper_1808_07217_amd import lsgd as L
    w = wk.get(name)
    cfg = L.make_config(w.widths, w.K, w.B_loc, w.N, dtype=w.dtype)
    assert L.param_count(cfg) == wk.param_count(w.widths)
    assert L.workspace_bytes(cfg) >= 2 * w.K * wk.param_count(w.widths) * 4


def test_known_parameter_counts():
    assert wk.param_count((64, 10)) == 650
    assert wk.param_count((3072, 512, 512, 10)) == 1841162
    assert wk.param_count((3072, 2048, 2048, 10)) == 10510346


@pytest.mark.parametrize("bad", [
    dict(K=0), dict(B_loc=0), dict(N=3, K=4), dict(widths=(64,)),
    dict(momentum=1.0), dict(momentum=-0.1), dict(weight_decay=-1.0),
    dict(widths=(64, 1)), dict(global_momentum=1.0),
    dict(global_momentum=-0.5), dict(global_momentum=float("nan")),
    dict(scheme=3), dict(scheme=-1), dict(scheme=1, global_momentum=0.5),
])
def test_invalid_configs_are_rejected(bad):
    from paper_1808_07217_amd import lsgd as L
    kw = dict(widths=(64, 10), K=4, B_loc=32, N=4096)
    kw.update(bad)
    opt = {k: kw.pop(k) for k in ("momentum", "weight_decay", "global_momentum")
           if k in kw}
    scheme = kw.pop("scheme", 0)
    if len(kw["widths"]) < 2:
        with pytest.raises(ValueError):
            L.make_config(**kw, **opt)
        return
    cfg = L.make_config(**kw, **opt)
    cfg.scheme = scheme
    with pytest.raises(L.LsgdError, match="invalid argument"):
        L.param_count(cfg)


def test_null_context_calls_fail_cleanly():
    from paper_1808_07217_amd import lsgd as L
    lib = L._lib
    assert lib.lsgd_average(None) == 1
    assert lib.lsgd_average_blocks(None, 1) == 1
    assert lib.lsgd_run_hierarchical_round(None, 1, 1, 1, None, None) == 1
    assert lib.lsgd_replica_average_blocks(None, 4, 2, 8, None) == 1
    assert lib.lsgd_synchronise(None, ctypes.c_float(0.1)) == 1
    assert lib.lsgd_read_error_memory(None, 0, None) == 1
    assert lib.lsgd_write_momentum(None, 0, None) == 1
    assert lib.lsgd_write_error_memory(None, 0, None) == 1
    assert lib.lsgd_replica_sign_sync(None, 4, 8, None, None, None, 0, None) == 1
    nb = ctypes.c_size_t()
    assert lib.lsgd_sign_sync_scratch_bytes(4, 6, ctypes.byref(nb)) == 1  # P % 4
    assert lib.lsgd_sign_sync_scratch_bytes(4, 8192, ctypes.byref(nb)) == 0
    # 2 bits per element, one fp64 partial per 8192-element chunk, K scales
    assert nb.value == 4 * 8192 * 2 // 8 + 256 + 256
    assert lib.lsgd_read_global_momentum(None, None) == 1
    assert lib.lsgd_write_global_momentum(None, None) == 1
    assert lib.lsgd_replica_average_global_momentum(
        None, 4, 8, None, None, ctypes.c_float(0.5), ctypes.c_float(0.1), None) == 1
    # a block size that does not divide K is refused before any launch
    fake = ctypes.c_void_p(256)
    assert lib.lsgd_replica_average_blocks(fake, 6, 4, 8, None) == 1
    assert lib.lsgd_replica_average_blocks(fake, 6, 0, 8, None) == 1
    # a global momentum factor outside [0, 1) or a zero step size likewise
    for mg, lr in ((1.0, 0.1), (-0.1, 0.1), (0.5, 0.0)):
        assert lib.lsgd_replica_average_global_momentum(
            fake, 4, 8, fake, fake, ctypes.c_float(mg), ctypes.c_float(lr), None) == 1
    assert lib.lsgd_local_step(None, ctypes.c_float(0.1), None) == 1
    assert lib.lsgd_destroy(None) == 1
    for s in range(7):
        assert lib.lsgd_status_string(s)
    assert lib.lsgd_last_error(None) == b""


def test_header_compiles_as_c99(tmp_path):
    """include/lsgd.h is a plain C99 header: a C translation unit that takes
    the address of every declared function compiles warning-free with
    -std=c99 -pedantic."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_lsgd.c"
    refs = "\n".join(f"  (void)&{n};" for n in _declared())
    src.write_text('#include "lsgd.h"\n#include <stdio.h>\n'
                   "int main(void) {\n"
                   "  lsgd_config cfg = {0};\n"
                   "  lsgd_status st = LSGD_E_NONFINITE;\n"
                   f"{refs}\n"
                   "  (void)cfg;\n"
                   "  printf(\"%d\\n\", (int)st);\n"
                   "  return 0;\n}\n")
    r = subprocess.run([cc, "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror",
                        "-I", os.path.join(ROOT, "include"), "-c", str(src), "-o",
                        str(tmp_path / "use_lsgd.o")], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _al(n):
    return (n + 255) // 256 * 256


@pytest.mark.parametrize("name,scheme,gm,sections", [
    ("resnet20", "local", 0.0, ("W", "U", "RS")),
    ("mlp_512", "local", 0.0, ("W", "U")),
    ("mlp_512", "ef_sign", 0.0, ("W", "U", "w_sync", "E")),
    ("mlp_512", "sign", 0.0, ("W", "U", "w_sync")),
    ("mlp_512", "local", 0.3, ("W", "U", "w_sync", "u_global")),
])
def test_state_blob_size_follows_the_documented_layout(name, scheme, gm, sections):
    """lsgd_state_bytes: a 256-byte header, then each present section at a
    256-byte aligned offset (replicas, momentum, BN running statistics of
    R = 2 x (16 x 7 + 32 x 6 + 64 x 6) = 1376 values, w_s, u, memories)."""
    from paper_1808_07217_amd import lsgd as L
    w = wk.get(name)
    cfg = L.make_config(w.widths, w.K, w.B_loc, w.N, dtype=w.dtype, model=w.model,
                        scheme=scheme, global_momentum=gm)
    K, P = w.K, L.param_count(cfg)
    R = 2 * (16 * 7 + 32 * 6 + 64 * 6)
    size = {"W": K * P, "U": K * P, "RS": K * R, "w_sync": P, "u_global": P, "E": K * P}
    assert L.state_bytes(cfg) == 256 + sum(_al(4 * size[s]) for s in sections)


def test_state_and_failure_calls_fail_cleanly():
    from paper_1808_07217_amd import lsgd as L
    lib = L._lib
    assert lib.lsgd_read_state(None, None) == 1
    assert lib.lsgd_write_state(None, None) == 1
    assert lib.lsgd_sync(None) == 1
    assert lib.lsgd_state_bytes(None, None) == 1
    assert lib.lsgd_status_string(6) == b"non-finite loss"


def test_resnet_batch_limit():
    """ResNet-20 batches must stay below 2^17 images per replica (each
    replica's largest activation then has fewer than 2^31 values)."""
    from paper_1808_07217_amd import lsgd as L
    ok = L.make_config((3072, 10), 2, (1 << 17) - 1, 4096, model="resnet20")
    assert L.param_count(ok) == 269722
    bad = L.make_config((3072, 10), 2, 1 << 17, 4096, model="resnet20")
    with pytest.raises(L.LsgdError, match="invalid argument"):
        L.param_count(bad)
