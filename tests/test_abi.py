"""The C ABI: the library loads without a GPU, exports every function the
header declares, and rejects invalid arguments on the host (no launch)."""

import ctypes
import os
import re
import subprocess

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "rbpolicy.h")


def _lib_path():
    from paper_2604_08706_amd import _binding

    if not os.path.exists(_binding.LIB_PATH):
        from paper_2604_08706_amd import build

        build.build(verbose=False)
    return _binding.LIB_PATH


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[\w]+\s*\**\s*(\w+)\s*\([^;]*\)\s*;", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("rb_sample_gather", "rb_group_advantage", "policy_logprob_fwd",
              "policy_loss_fwd_bwd", "policy_logprob_bwd", "rbp_workspace_bytes",
              "rbp_status_string", "rbp_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    path = _lib_path()
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [n for n in _declared_functions() if n not in exported]
    assert not missing, missing
    lib = ctypes.CDLL(path)
    for n in _declared_functions():
        assert getattr(lib, n) is not None


def test_binding_names_match_header():
    from paper_2604_08706_amd import _binding

    assert sorted(_binding.EXPORTED) == _declared_functions()


def test_status_strings_and_workspace_sizes():
    from paper_2604_08706_amd import _binding as b

    lib = b.load_library(_lib_path())
    assert lib.rbp_status_string(0) == b"ok"
    assert lib.rbp_status_string(-3) == b"workspace too small"
    assert lib.rbp_status_string(12345) == b"unknown status"
    assert lib.rbp_workspace_bytes(99, 10, 8, 8) == 0
    # backward workspace: dz^T bf16 [Vp, Tc] and the second dhidden K half
    # fp32 [Tc, d] (Tc and Vp rounded up to 256)
    assert lib.rbp_workspace_bytes(b.RBP_OP_LOGPROB_BWD, 16384, 3584, 152064) == \
        152064 * 16384 * 2 + 16384 * 3584 * 4
    assert lib.rbp_workspace_bytes(b.RBP_OP_LOGPROB_BWD, 1, 64, 1000) == \
        1024 * 256 * 2 + 256 * 64 * 4
    # forward workspace: one (max, sum) pair per 128-row half of each vocab
    # tile and token (tokens rounded up to 256)
    assert lib.rbp_workspace_bytes(b.RBP_OP_LOGPROB_FWD, 100, 64, 513) == 256 * 6 * 8
    assert lib.rbp_workspace_bytes(b.RBP_OP_LOSS, 10, 0, 0) > 0
    # fused workspace: exp(z - R) bf16 [Vp, Tc], (max, sum, sum z) fp32
    # [Vp / 128, Tc] each, five per-token arrays [Tc] (target logit, R,
    # reference, scale, list) and the list's count, the scaled hidden states
    # bf16 [Tc, d], the dhidden K half and the loss pass's sums
    loss = lib.rbp_workspace_bytes(b.RBP_OP_LOSS, 16384, 0, 0)
    assert lib.rbp_workspace_bytes(b.RBP_OP_FUSED, 16384, 3584, 152064) == \
        152064 * 16384 * 2 + 3 * 1188 * 16384 * 4 + 5 * 16384 * 4 + 256 + \
        16384 * 3584 * 2 + 16384 * 3584 * 4 + (loss + 255) // 256 * 256
    assert lib.rbp_workspace_bytes(b.RBP_OP_SAMPLE_GATHER, 1_000_000, 0, 0) >= 4_000_000


def test_invalid_arguments_fail_on_the_host():
    from paper_2604_08706_amd import _binding as b

    lib = b.load_library(_lib_path())
    null = ctypes.c_void_p(0)
    assert lib.rb_sample_gather(None, None, None, null, 0, null) == b.RBP_EINVAL
    assert b"null" in lib.rbp_last_error()
    rec = b.RbRecords()
    rec.n_live, rec.capacity, rec.head = 5, 4, 0  # n_live > capacity
    cfg = b.RbSampleCfg()
    out = b.RbBatch()
    assert lib.rb_sample_gather(ctypes.byref(rec), ctypes.byref(cfg), ctypes.byref(out), null, 0,
                                null) == b.RBP_EINVAL
    assert lib.policy_logprob_fwd(null, null, null, null, -1, 64, 10, null, null, null, 0,
                                  null) == b.RBP_EINVAL
    assert lib.policy_logprob_fwd(null, null, null, null, 4, 12, 10, null, null, null, 0,
                                  null) == b.RBP_EUNSUPPORTED
    assert lib.policy_logprob_bwd(null, null, null, null, null, null, 4, 12, 10, null, null, 0,
                                  null, 0, null) == b.RBP_EUNSUPPORTED
    assert lib.policy_loss_fwd_bwd(null, null, null, null, null, 4, 0, 1, 0.2, 0.2, null, null,
                                   null, null, 0, null) == b.RBP_EINVAL
    assert lib.rb_group_advantage(null, null, 3, 1, 1e-6, null, null) == b.RBP_EINVAL
    assert lib.rb_group_advantage(ctypes.c_void_p(8), ctypes.c_void_p(8), 3, 2, 1e-6,
                                  ctypes.c_void_p(8), null) == b.RBP_EINVAL
    assert lib.rb_hist_accumulate(null, 5, 0, 4, null, null) == b.RBP_EINVAL
    assert lib.rb_hist_accumulate(null, 0, 0, 0, null, null) == b.RBP_EINVAL
    assert lib.rb_hist_accumulate(null, 0, 0, 4097, null, null) == b.RBP_EINVAL
    # a replay-ratio histogram needs the use counts
    ring = b.RbRing()
    ring.capacity, ring.slot_tokens = 4, 2
    for f in ("arena_off", "length", "reward", "advantage", "version", "arena_tokens",
              "arena_old_logp", "replay_hist"):
        setattr(ring, f, 8)
    ring.replay_bins = 4
    d8 = ctypes.c_void_p(8)
    assert lib.rb_push(ctypes.byref(ring), 2, 1, d8, d8, d8, d8, 0, d8, d8, 1, 1e-6,
                       null) == b.RBP_EINVAL
    assert b"replay_hist" in lib.rbp_last_error()
    lib.rbp_status_string(0)
    # a successful call clears the thread's error text
    assert lib.rb_group_advantage(ctypes.c_void_p(8), ctypes.c_void_p(8), 0, 1, 1e-6,
                                  ctypes.c_void_p(8), null) == b.RBP_OK
    assert lib.rbp_last_error() == b""


def test_product_path_fails_loudly_without_the_library(tmp_path):
    from paper_2604_08706_amd import _binding as b

    with pytest.raises(ImportError):
        b.load_library(str(tmp_path / "missing.so"))


C_CLIENT = r"""
#include <stdio.h>
#include <string.h>
#include "rbpolicy.h"

int main(void) {
  /* workspace sizes are host arithmetic: dz^T bf16 [Vp][Tc] + fp32 [Tc][d] */
  const size_t want = (size_t)152064 * 16384 * 2 + (size_t)16384 * 3584 * 4;
  if (rbp_workspace_bytes(RBP_OP_LOGPROB_BWD, 16384, 3584, 152064) != want) return 1;
  /* invalid arguments are rejected on the host, before any launch */
  if (rb_group_advantage(NULL, NULL, 3, 1, 1e-6f, NULL, NULL) != RBP_EINVAL) return 2;
  if (strlen(rbp_last_error()) == 0) return 3;
  if (policy_logprob_fwd(NULL, NULL, NULL, NULL, 4, 12, 10, NULL, NULL, NULL, 0, NULL) !=
      RBP_EUNSUPPORTED) return 4;
  if (strcmp(rbp_status_string(RBP_OK), "ok") != 0) return 5;
  printf("c client ok\n");
  return 0;
}
"""


def test_header_compiles_as_c99_and_links(tmp_path):
    """A plain C99 client (gcc, -pedantic -Werror) includes the header, links
    the library and calls host-side entry points: the boundary needs no C++
    and no torch."""
    import shutil

    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("needs gcc")
    lib = _lib_path()
    src = tmp_path / "client.c"
    src.write_text(C_CLIENT)
    exe = tmp_path / "client"
    libdir = os.path.dirname(lib)
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                    "-L", libdir, "-lrbpolicy", "-Wl,-rpath," + libdir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "c client ok" in r.stdout
