"""C-ABI checks that need no GPU: libpair.so loads, exports every entry point
declared in include/pair.h, and rejects malformed arguments on the host
before anything is enqueued (these calls never reach the HIP runtime)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2608_11368_amd as pair

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pair.h")

FAKE = ctypes.c_void_p(1 << 20)           # 16-byte aligned non-null stand-in, never dereferenced
ODD = ctypes.c_void_p((1 << 20) + 2)      # misaligned stand-in
NULL = None


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|size_t|const char\*)\s+(pair_\w+)\(", src, re.M)))


def test_header_declares_the_four_calls():
    names = _declared()
    for n in ("pair_design_inclusion", "pair_edge_coeffs", "pair_weighted_grad", "pair_audit"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = pair.lib()
    names = _declared()
    assert names
    for n in names:
        assert hasattr(L, n), n
    dyn = subprocess.run(["nm", "-D", "--defined-only", pair.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s+(pair_\w+)$", dyn, re.M))
    assert set(names) <= exported
    assert set(pair.EXPORTED) == set(names)


def test_version_and_strerror():
    assert pair.version() >= 100
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -99):
        assert isinstance(pair.strerror(code), str) and pair.strerror(code)


def test_design_inclusion_rejects_bad_arguments():
    L = pair.lib()
    f = L.pair_design_inclusion
    ok = dict(B=4, nv=32, gmax=8, offsets=FAKE, p=FAKE, seed=1, rep0=0, R=1, mask=FAKE, pi=NULL,
              ec=NULL, comp=NULL, st=NULL, stream=NULL)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["B"], a["nv"], a["gmax"], a["offsets"], a["p"], a["seed"], a["rep0"], a["R"],
                 a["mask"], a["pi"], a["ec"], a["comp"], a["st"], a["stream"])

    assert call(offsets=NULL) == -1
    assert call(p=NULL) == -1
    assert call(B=0) == -1
    assert call(gmax=1) == -3
    assert call(gmax=65) == -3
    assert call(R=0) == -3
    assert call(rep0=-1) == -3
    assert call(mask=NULL) == -1          # nothing to produce


def test_edge_coeffs_rejects_bad_arguments():
    f = pair.lib().pair_edge_coeffs
    assert f(4, 32, 8, NULL, FAKE, NULL, NULL, FAKE, NULL, NULL, NULL) == -1
    assert f(4, 32, 8, FAKE, NULL, NULL, NULL, FAKE, NULL, NULL, NULL) == -1
    assert f(4, 32, 8, FAKE, FAKE, NULL, NULL, NULL, NULL, NULL, NULL) == -1
    assert f(4, 32, 100, FAKE, FAKE, NULL, NULL, FAKE, NULL, NULL, NULL) == -3
    assert f(-1, 32, 8, FAKE, FAKE, NULL, NULL, FAKE, NULL, NULL, NULL) == -1


def test_weighted_grad_rejects_bad_arguments():
    f = pair.lib().pair_weighted_grad

    def call(B=4, nv=32, off=FAKE, D=64, s=FAKE, dt=1, ld=64, c=FAKE, out=FAKE, reduce=0):
        return f(B, nv, off, D, s, dt, ld, c, out, reduce, NULL, NULL)

    assert call(off=NULL) == -1
    assert call(s=NULL) == -1
    assert call(c=NULL) == -1
    assert call(out=NULL) == -1
    assert call(reduce=2) == -1
    assert call(reduce=-1) == -1
    assert call(dt=7) == -2
    assert call(D=0) == -3
    assert call(ld=63) == -3
    assert call(s=ODD) == -4
    assert call(ld=66) == -4              # bf16 rows of 132 bytes are not 16-byte aligned
    assert call(dt=0, ld=66) == -4        # fp32 rows of 264 bytes are not 16-byte aligned


def test_audit_rejects_bad_arguments_and_sizes_workspace():
    L = pair.lib()
    need = L.pair_audit_workspace_bytes(256, 16, 65536, 4096)
    assert need > 256 * 4096 * 16 * 2                     # bf16 deviations at least
    assert L.pair_audit_workspace_bytes(4, 65, 64, 10) == 0
    assert L.pair_audit_workspace_bytes(4, 8, 64, 0) == 0
    f = L.pair_audit

    def call(dt=1, ws=FAKE, wsb=need, R=4096, gmax=16, mse=FAKE, s=FAKE):
        return f(256, 4096, gmax, FAKE, 65536, s, dt, 65536, FAKE, FAKE, NULL, 1, 0, R, mse, FAKE,
                 NULL, NULL, ws, wsb, NULL, NULL)

    assert call(dt=0) == -2               # the matrix-core path takes bf16 scores
    assert call(ws=NULL) == -6
    assert call(wsb=need - 1) == -6
    assert call(ws=ctypes.c_void_p((1 << 20) + 16)) == -6   # workspace must be 256-byte aligned
    assert call(R=0) == -3
    assert call(gmax=80) == -3
    assert call(mse=NULL) == -1
    assert call(s=ODD) == -4


def test_audit_noalloc_rejects_bad_arguments_and_oversized_prompts():
    L = pair.lib()
    f = L.pair_audit_noalloc

    def call(dt=1, R=4096, gmax=16, mse=FAKE, s=FAKE, D=65536, rep0=0):
        return f(256, 4096, gmax, FAKE, D, s, dt, D, FAKE, FAKE, NULL, 1, rep0, R, mse, FAKE,
                 NULL, NULL, NULL, NULL)

    assert call(dt=0) == -2
    assert call(R=0) == -3
    assert call(rep0=-1) == -3
    assert call(gmax=80) == -3
    assert call(mse=NULL) == -1
    assert call(s=ODD) == -4
    # one prompt of 16 candidates, 2^23 score columns and 4096 replicates needs
    # more workspace than the static scratch holds: rejected before any HIP call
    assert L.pair_audit_workspace_bytes(1, 16, 1 << 23, 4096) > pair.AUDIT_SCRATCH_BYTES
    assert call(D=1 << 23) == -7
    assert "scratch" in pair.strerror(-7)


def test_design_alloc_ex_rejects_bad_arguments():
    f = pair.lib().pair_design_alloc_ex

    def call(B=4, gmax=8, off=FAKE, pi=FAKE, design=0, pi_min=0.08, max_sweeps=0):
        return f(B, 32, gmax, off, FAKE, FAKE, NULL, FAKE, pi_min, design, NULL, max_sweeps, pi,
                 NULL, NULL, NULL, NULL, NULL)

    assert call(off=NULL) == -1
    assert call(pi=NULL) == -1
    assert call(B=0) == -1
    assert call(gmax=65) == -3
    assert call(design=3) == -1
    assert call(pi_min=0.0) == -3
    assert call(max_sweeps=-1) == -3


def test_binding_checks_tensors_before_calling():
    import torch

    t = torch.zeros(4)
    with pytest.raises(ValueError):
        pair._dev(t, "x", torch.float32)          # host tensor is refused


def test_rule_entry_points_reject_bad_rules():
    L = pair.lib()
    f = L.pair_edge_coeffs_rule

    def call(rule=0, wmax=0.0, rewards=FAKE, coeff=FAKE):
        return f(4, 32, 8, FAKE, rewards, NULL, NULL, rule, wmax, coeff, NULL, NULL, NULL, NULL,
                 NULL)

    assert call(rule=6) == -1
    assert call(rule=-1) == -1
    assert call(rule=pair.RULE_CLIPPED, wmax=0.0) == -1
    assert call(rule=pair.RULE_CLIPPED, wmax=-2.0) == -1
    assert call(rule=pair.RULE_CLIPPED, wmax=float("inf")) == -1
    assert call(rule=pair.RULE_CLIPPED, wmax=float("nan")) == -1
    assert call(rewards=NULL) == -1
    assert call(coeff=NULL) == -1
    need = L.pair_audit_workspace_bytes(4, 8, 64, 10)
    g = L.pair_audit_rule

    def acall(rule=0, wmax=0.0):
        return g(4, 32, 8, FAKE, 64, FAKE, 1, 64, FAKE, FAKE, NULL, rule, wmax, 1, 0, 10, FAKE,
                 FAKE, NULL, NULL, FAKE, need, NULL, NULL)

    assert acall(rule=7) == -1
    assert acall(rule=pair.RULE_CLIPPED, wmax=0.0) == -1


def test_audit_direction_rejects_bad_arguments_and_sizes_workspace():
    L = pair.lib()
    need = L.pair_audit_direction_workspace_bytes(256, 16, 65536, 4096)
    assert need > 256 * 4096 * 16 * 4                     # fp32 deviations at least
    assert L.pair_audit_direction_workspace_bytes(4, 65, 64, 10) == 0
    assert L.pair_audit_direction_workspace_bytes(4, 8, 64, 0) == 0
    assert L.pair_audit_direction_workspace_bytes(4, 8, 0, 10) == 0
    f = L.pair_audit_direction

    def call(dt=1, ws=FAKE, wsb=need, R=4096, gmax=16, cos=FAKE, tn=FAKE, s=FAKE, rule=0,
             wmax=0.0, rep0=0):
        return f(256, 4096, gmax, FAKE, 65536, s, dt, 65536, FAKE, FAKE, NULL, rule, wmax, 1, rep0,
                 R, cos, tn, ws, wsb, NULL, NULL)

    assert call(dt=0) == -2
    assert call(ws=NULL) == -6
    assert call(wsb=need - 1) == -6
    assert call(ws=ctypes.c_void_p((1 << 20) + 16)) == -6
    assert call(R=0) == -3
    assert call(rep0=-1) == -3
    assert call(gmax=80) == -3
    assert call(cos=NULL) == -1
    assert call(tn=NULL) == -1
    assert call(rule=9) == -1
    assert call(rule=pair.RULE_CLIPPED, wmax=0.0) == -1
    assert call(s=ODD) == -4


def test_header_is_plain_c_and_links_from_a_c_caller(tmp_path):
    """include/pair.h compiles as strict C99 and as C++11, and a C program
    linked against libpair.so runs the host-side entry points (no GPU: the
    calls it makes return before touching the device)."""
    prog = tmp_path / "caller.c"
    prog.write_text(r'''
#include <stdio.h>
#include <string.h>
#include "pair.h"
int main(void) {
  if (pair_version() < 100) return 1;
  if (strcmp(pair_strerror(PAIR_OK), "ok") != 0) return 2;
  /* argument checks happen before any device work */
  if (pair_weighted_grad(4, 32, NULL, 64, NULL, PAIR_BF16, 64, NULL, NULL, 0, NULL, NULL) !=
      PAIR_EINVAL) return 3;
  if (pair_audit_workspace_bytes(4, 65, 64, 10) != 0) return 4;
  printf("c caller ok %d\n", pair_version());
  return 0;
}
''')
    inc = os.path.join(ROOT, "include")
    for cmd in (["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-fsyntax-only"],
                ["g++", "-std=c++11", "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-x", "c++"]):
        subprocess.run(cmd + ["-I", inc, str(prog)], check=True, capture_output=True)
    libdir = os.path.dirname(pair.LIB_PATH)
    exe = tmp_path / "caller"
    subprocess.run(["gcc", "-std=c99", "-I", inc, str(prog), "-o", str(exe), "-L", libdir,
                    "-l:" + os.path.basename(pair.LIB_PATH), f"-Wl,-rpath,{libdir}",
                    "-Wl,-rpath-link,/opt/rocm/lib"], check=True, capture_output=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "c caller ok" in res.stdout
