"""Register and scratch budgets of the hot kernels, from the compiler's
resource report for gfx950 (CPU only: hipcc cross-compiles without a GPU).

* No kernel may spill to scratch: a spill in a 256 x 256 tile kernel costs
  gigabytes of scratch traffic per launch.
* The tile kernels run two waves per SIMD: at most 256 VGPRs each.
"""

import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2604_08706_amd import build as b

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None and
                                not os.path.exists("/opt/rocm/bin/hipcc"),
                                reason="needs hipcc")

_REPORT = {}


def _resources(src):
    """{kernel name fragment: (vgprs, scratch bytes per lane)} for one source."""
    if src in _REPORT:
        return _REPORT[src]
    with tempfile.TemporaryDirectory() as tmp:
        cmd = [b.hipcc(), *b.FLAGS, "-Rpass-analysis=kernel-resource-usage", "-c",
               os.path.join(b.CSRC, src), "-o", os.path.join(tmp, "k.o")]
        r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out, name = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            out[name] = [None, None]
        m = re.search(r"VGPRs: (\d+)", line)
        if m and name:
            out[name][0] = int(m.group(1))
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            out[name][1] = int(m.group(1))
    _REPORT[src] = out
    return out


def _kernels(src, fragment):
    """Every instance (template instantiations included) of a kernel."""
    hits = [v for k, v in _resources(src).items() if fragment in k]
    assert hits, (src, fragment, list(_resources(src)))
    return hits


@pytest.mark.parametrize("src,kernel", [
    ("logprob_fwd.hip", "logits_lse_partial_kernel"),
    ("logprob_bwd.hip", "grad_logits_kernel"),
    ("logprob_bwd.hip", "dhidden_kernel"),
    ("logprob_bwd.hip", "dhidden_pieces_kernel"),
    ("logprob_bwd.hip", "dweight_kernel"),
    ("fused.hip", "logits_store_kernel"),
    ("fused.hip", "fused_merge_kernel"),
    ("fused.hip", "fixup_kernel"),
    ("fused.hip", "token_scale_kernel"),
    ("sample_gather.hip", "select_rest_kernel"),
    ("sample_gather.hip", "draw_kernel"),
])
def test_hot_kernels_do_not_spill(src, kernel):
    for vgprs, scratch in _kernels(src, kernel):
        assert scratch == 0, f"{kernel} spills {scratch} bytes per lane"
        assert vgprs <= 256
