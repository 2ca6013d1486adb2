"""Host-side checks of the C ABI library (no GPU needed): it loads, exports
every entry point that include/zo.h declares, its host-only functions agree
with the oracle's layout, and argument errors are reported before anything
touches a device."""
import ctypes as C
import os
import re

import pytest

from paper_2505_17852_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zo.h")


@pytest.fixture(scope="module")
def zo():
    from paper_2505_17852_amd import zo as z
    if not os.path.exists(z.LIB_PATH):
        from paper_2505_17852_amd import build
        build.build()
    z.lib()
    return z


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(zo_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_step(zo):
    names = declared_symbols()
    for n in ("zo_init", "zo_perturbed_losses", "zo_update", "zo_param_count",
              "zo_workspace_bytes", "zo_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(zo):
    L = zo.lib()
    for n in declared_symbols():
        assert hasattr(L, n), n


@pytest.mark.parametrize("name", wl.CONFIG_ORDER)
def test_param_count_matches_oracle_layout(zo, oracle, name):
    cfg = wl.model_cfg(name)
    assert zo.param_count(cfg) == oracle.param_count(cfg) == wl.param_count(cfg)


def test_param_count_closed_form_values(zo):
    # closed-form counts of the five workloads
    expect = {"c1": 49_664, "c2": 1_018_112, "c3": 127_628_112, "c4": 1_215_054_672,
              "c5": 3_354_880}
    for name, p in expect.items():
        assert zo.param_count(wl.model_cfg(name)) == p


def test_workspace_bytes(zo):
    cfg = wl.model_cfg("c2")
    n = zo.workspace_bytes(cfg, 32, 64, 256)
    assert n > 0
    assert zo.workspace_bytes(cfg, 64, 64, 256) > n
    assert zo.workspace_bytes(cfg, 0, 64, 256) == 0
    bad = dict(cfg, n_layers=0)
    assert zo.workspace_bytes(bad, 4, 4, 4) == 0
    assert zo.workspace_bytes_min(bad, 4, 4, 4) == 0


@pytest.mark.parametrize("name", wl.CONFIG_ORDER)
def test_workspace_probe_cache_size(zo, name):
    """Normal probes: the preferred workspace adds exactly the probe cache,
    N values of the weight matrices' size in the weight type (rounded up to
    the 256-byte allocation granule; with bf16 weights the head matrix is
    stored padded to whole 256-wide vocabulary tiles, and each probe has two
    blocks: its perturbed weights for +eps and -eps); sign probes with bf16
    weights add the sign-probe cache, with fp32 weights nothing."""
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    full = zo.workspace_bytes(cfg, w["N"], w["B"], w["C"])
    small = zo.workspace_bytes_min(cfg, w["N"], w["B"], w["C"])
    if cfg["probe"] == wl.GAUSSIAN:
        L, E, H, V = cfg["n_layers"], cfg["embed"], cfg["hidden"], cfg["vocab"]
        # bf16: the head matrix is stored padded to whole 256-wide vocabulary tiles
        Vs = (V + 255) // 256 * 256 if cfg["wdtype"] == wl.BF16 else V
        pg = sum(4 * H * ((E if l == 0 else H) + H) for l in range(L)) + Vs * H
        el = 2 * 2 if cfg["wdtype"] == wl.BF16 else 4
        assert full - small == (w["N"] * pg * el + 255) // 256 * 256
    elif cfg["wdtype"] == wl.BF16:
        # sign probes with bf16 weights: the sign-probe cache, N words of 32 signs per 32 parameters
        P = zo.param_count(cfg)
        words = (P + 127) // 128 * 4
        assert full - small == (w["N"] * words * 4 + 255) // 256 * 256
        assert zo.lib().zo_probe_bits_offset(C.byref(zo._cfg(cfg)), w["N"], w["B"], w["C"]) == small
    else:
        assert full == small
        assert zo.lib().zo_probe_bits_offset(C.byref(zo._cfg(cfg)), w["N"], w["B"], w["C"]) == 0


def test_update_cached_argument_errors(zo):
    """zo_update_cached takes sign probes only and checks its pointers on the
    host; zo_probe_bits_offset is 0 without a cache."""
    L = zo.lib()
    fake = C.c_void_p(0x10000)
    bf = zo._cfg(dict(n_layers=1, vocab=256, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.RADEMACHER))
    gauss = zo._cfg(dict(n_layers=1, vocab=256, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.GAUSSIAN))
    assert L.zo_update_cached(C.byref(gauss), fake, 1, 1e-3, 1e-3, 2, 0, fake, fake, None, fake, None) == zo.ZO_EINVAL
    assert L.zo_update_cached(C.byref(bf), fake, 1, 1e-3, 1e-3, 2, 0, fake, fake, None, None, None) == zo.ZO_EINVAL
    assert L.zo_update_cached(C.byref(bf), fake, 1, 1e-3, 1e-3, 2, 0, fake, fake, None, C.c_void_p(0x10004),
                              None) == zo.ZO_EINVAL
    assert L.zo_update_cached(C.byref(bf), fake, 1, 0.0, 1e-3, 2, 0, fake, fake, None, fake, None) == zo.ZO_EINVAL
    assert L.zo_probe_bits_offset(C.byref(gauss), 2, 2, 2) == 0
    assert L.zo_probe_bits_offset(C.byref(bf), 0, 2, 2) == 0
    assert L.zo_probe_bits_offset(C.byref(bf), 2, 2, 2) > 0


def _call_losses(zo, cfg, eps=1e-3, N=2, B=2, Cn=4, ptrs=True):
    c = zo._cfg(cfg)
    fake = C.c_void_p(0x10000) if ptrs else None
    return zo.lib().zo_perturbed_losses(C.byref(c), fake, 1, eps, N, 0, fake, None, B, Cn,
                                        fake, fake, fake, 1 << 40, None)


def test_argument_errors_before_any_device_work(zo):
    cfg = wl.model_cfg("c1")
    assert _call_losses(zo, dict(cfg, n_layers=0)) == zo.ZO_EINVAL
    assert _call_losses(zo, dict(cfg, probe=7)) == zo.ZO_EINVAL
    assert _call_losses(zo, dict(cfg, hidden=48)) == zo.ZO_ESHAPE
    assert _call_losses(zo, dict(cfg, embed=20)) == zo.ZO_ESHAPE
    assert _call_losses(zo, dict(cfg, wdtype=1, hidden=96)) == zo.ZO_ESHAPE  # bf16: K tiles of 64
    assert _call_losses(zo, cfg, eps=0.0) == zo.ZO_EINVAL
    assert _call_losses(zo, cfg, eps=float("nan")) == zo.ZO_EINVAL
    assert _call_losses(zo, cfg, N=0) == zo.ZO_EINVAL
    assert _call_losses(zo, cfg, B=0) == zo.ZO_EINVAL
    assert _call_losses(zo, cfg, ptrs=False) == zo.ZO_EINVAL
    assert "NULL" in zo.lib().zo_last_error().decode()
    c = zo._cfg(cfg)
    fake = C.c_void_p(0x10000)
    ws_small = zo.lib().zo_perturbed_losses(C.byref(c), fake, 1, 1e-3, 2, 0, fake, None, 2, 4,
                                            fake, fake, fake, 16, None)
    assert ws_small == zo.ZO_ENOMEM
    L = zo.lib()
    assert L.zo_update(C.byref(c), fake, 1, 1e-3, float("inf"), 2, 0, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_update(C.byref(c), fake, 1, -1.0, 1e-3, 2, 0, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_update(C.byref(c), fake, 1, 1e-3, 1e-3, 0, 0, fake, fake, None, None) == zo.ZO_EINVAL
    # probe indices must stay within 32 bits
    assert L.zo_update(C.byref(c), fake, 1, 1e-3, 1e-3, 4, 0xFFFFFFFE, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_debug_probe(5, 1, 0, 0, 4, fake, None) == zo.ZO_EINVAL


def test_forward_difference_argument_errors(zo):
    """zo_fd_losses and zo_fd_update validate like their central-difference
    counterparts, before anything touches the device."""
    cfg = wl.model_cfg("c1")
    c = zo._cfg(cfg)
    fake = C.c_void_p(0x10000)
    L = zo.lib()

    def fd_losses(eps=1e-3, N=2, B=2, Cn=4, i0=0, ws=1 << 40, theta=fake, cfgv=c):
        return L.zo_fd_losses(C.byref(cfgv), theta, 1, eps, N, i0, fake, None, B, Cn, fake, fake, fake, ws, None)

    assert fd_losses(eps=0.0) == zo.ZO_EINVAL
    assert fd_losses(eps=float("inf")) == zo.ZO_EINVAL
    assert fd_losses(N=0) == zo.ZO_EINVAL
    assert fd_losses(B=0) == zo.ZO_EINVAL
    assert fd_losses(Cn=0) == zo.ZO_EINVAL
    assert fd_losses(N=3, i0=0xFFFFFFFE) == zo.ZO_EINVAL
    assert fd_losses(theta=None) == zo.ZO_EINVAL
    assert fd_losses(theta=C.c_void_p(0x10004)) == zo.ZO_EINVAL  # theta not 16-byte aligned
    assert fd_losses(ws=16) == zo.ZO_ENOMEM
    assert fd_losses(cfgv=zo._cfg(dict(cfg, hidden=40))) == zo.ZO_ESHAPE
    assert L.zo_fd_update(C.byref(c), fake, 1, 1e-3, float("nan"), 2, 0, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_fd_update(C.byref(c), fake, 1, 0.0, 1e-3, 2, 0, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_fd_update(C.byref(c), fake, 1, 1e-3, 1e-3, 0, 0, fake, fake, None, None) == zo.ZO_EINVAL
    assert L.zo_fd_update(C.byref(c), fake, 1, 1e-3, 1e-3, 2, 0, fake, None, None, None) == zo.ZO_EINVAL
    assert L.zo_fd_update(C.byref(c), fake, 1, 1e-3, 1e-3, 4, 0xFFFFFFFE, fake, fake, None, None) == zo.ZO_EINVAL


def test_products_and_eps_floor_errors(zo):
    """The form of the products and the bf16 eps floor are checked on the
    host: bf16 weights reject eps below ZO_BF16_EPS_MIN (2^-17) and accept it
    at the floor (the call then fails only on the 16-byte workspace);
    unknown product forms and the fp32 two-stream form of forward differences
    are argument errors."""
    L = zo.lib()
    fake = C.c_void_p(0x10000)
    bf = zo._cfg(dict(n_layers=1, vocab=256, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.RADEMACHER))
    f32 = zo._cfg(wl.model_cfg("c1"))

    def losses(cfgv, eps, products=zo.PRODUCTS_AUTO, ws=1 << 40, fd=False):
        f = L.zo_fd_losses_ex if fd else L.zo_perturbed_losses_ex
        return f(C.byref(cfgv), fake, 1, eps, 2, 0, fake, None, 2, 4, fake, fake, fake, ws, products, None)

    assert losses(bf, 2.0 ** -18) == zo.ZO_EINVAL
    assert "eps" in L.zo_last_error().decode()
    assert losses(bf, 2.0 ** -17, ws=16) == zo.ZO_ENOMEM
    assert losses(bf, 2.0 ** -18, products=zo.PRODUCTS_SPLIT) == zo.ZO_EINVAL
    assert L.zo_perturbed_losses(C.byref(bf), fake, 1, 2.0 ** -18, 2, 0, fake, None, 2, 4, fake, fake, fake,
                                 1 << 40, None) == zo.ZO_EINVAL
    assert L.zo_fd_losses(C.byref(bf), fake, 1, 2.0 ** -18, 2, 0, fake, None, 2, 4, fake, fake, fake,
                          1 << 40, None) == zo.ZO_EINVAL
    assert losses(f32, 2.0 ** -20, ws=16) == zo.ZO_ENOMEM  # fp32 weights have no floor
    assert losses(bf, 1e-3, products=3) == zo.ZO_EINVAL
    assert losses(bf, 1e-3, products=-1) == zo.ZO_EINVAL
    assert losses(f32, 1e-3, products=zo.PRODUCTS_SPLIT, fd=True) == zo.ZO_EINVAL
    assert losses(f32, 1e-3, products=zo.PRODUCTS_SPLIT, ws=16) == zo.ZO_ENOMEM
    assert losses(bf, 1e-3, products=zo.PRODUCTS_SPLIT, ws=16, fd=True) == zo.ZO_ENOMEM
    assert zo.BF16_EPS_MIN == 2.0 ** -17 and zo.BF16_FUSED_EPS_MIN == 2.0 ** -10


def test_noalloc_size_check_on_the_host(zo):
    """zo_perturbed_losses_noalloc rejects a shape whose workspace exceeds its
    fixed scratch (ZO_ENOMEM) and bad sizes (ZO_EINVAL) before any device
    work; the c1 and c2 workloads fit the scratch, the billion-parameter ones
    do not."""
    L = zo.lib()
    fake = C.c_void_p(0x10000)
    for name in ("c1", "c2"):
        w = wl.CONFIGS[name]
        assert zo.workspace_bytes_min(wl.model_cfg(name), w["N"], w["B"], w["C"]) <= zo.NOALLOC_WORKSPACE_BYTES
    for name in ("c3", "c4", "c5"):
        w = wl.CONFIGS[name]
        c = zo._cfg(wl.model_cfg(name))
        assert zo.workspace_bytes_min(wl.model_cfg(name), w["N"], w["B"], w["C"]) > zo.NOALLOC_WORKSPACE_BYTES
        assert L.zo_perturbed_losses_noalloc(C.byref(c), fake, 1, 1e-3, w["N"], 0, fake, None, w["B"], w["C"],
                                             fake, fake, None) == zo.ZO_ENOMEM
        assert "scratch" in L.zo_last_error().decode()
    c = zo._cfg(wl.model_cfg("c1"))
    assert L.zo_perturbed_losses_noalloc(C.byref(c), fake, 1, 1e-3, 0, 0, fake, None, 4, 32, fake, fake,
                                         None) == zo.ZO_EINVAL


def test_header_is_c_and_the_library_links_from_c(zo, tmp_path):
    """include/zo.h compiles as C11, and a C program linked against the
    library calls its host-only entry points (sizes and argument checks; no
    device work) and reads the same numbers as the binding."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.dirname(zo.LIB_PATH)
    src = tmp_path / "abi.c"
    src.write_text(r'''
#include <stdio.h>
#include "zo.h"
int main(void) {
    zo_config c = {1, 256, 32, 64, ZO_WFP32, ZO_RADEMACHER};
    zo_config bad = {0, 256, 32, 64, ZO_WFP32, ZO_RADEMACHER};
    printf("%zu %zu %zu %zu\n", zo_param_count(&c), zo_workspace_bytes(&c, 8, 4, 32),
           zo_workspace_bytes_min(&c, 8, 4, 32), zo_param_count(&bad));
    int st = zo_update(&c, NULL, 1, 1e-3f, 1e-3f, 8, 0, NULL, NULL, NULL, NULL);
    printf("%d %s\n", st, zo_last_error());
    return 0;
}
''')
    exe = tmp_path / "abi"
    subprocess.run([gcc, "-std=c11", "-Wall", "-Werror", "-I", os.path.join(root, "include"), str(src),
                    "-L", libdir, "-l:" + os.path.basename(zo.LIB_PATH), "-Wl,-rpath," + libdir, "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    cfg = wl.model_cfg("c1")
    p, ws, wsmin, zero = (int(x) for x in out[0].split())
    assert p == zo.param_count(cfg) and zero == 0
    assert ws == zo.workspace_bytes(cfg, 8, 4, 32) and wsmin == zo.workspace_bytes_min(cfg, 8, 4, 32)
    st, msg = out[1].split(" ", 1)
    assert int(st) == zo.ZO_EINVAL and "NULL" in msg
