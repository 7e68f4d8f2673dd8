"""The library loaded before torch in a fresh process (the binding imports
torch first, so the process holds torch's HIP runtime only): a forward call
there succeeds and matches the same call in this process bit for bit.
Without that order the process held two HIP runtimes and every call failed
with GS_ERR_HIP."""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
from paper_2609_04910_amd import gauss_sum as gs
gs.load()
import torch
rng = np.random.default_rng(3)
q = torch.from_numpy(rng.standard_normal((300, 24)).astype(np.float16)).cuda()
k = torch.from_numpy(rng.standard_normal((500, 24)).astype(np.float16)).cuda()
v = torch.from_numpy(rng.standard_normal((500, 5)).astype(np.float32)).cuda()
s = gs.gauss_sum_fwd(q, k, v, 0.05)
torch.cuda.synchronize()
np.save(sys.argv[2], s.cpu().numpy())
print("child ok", flush=True)
"""


def test_library_loaded_before_torch(tmp_path):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    gs.load()
    out = str(tmp_path / "child.npy")
    print("child process: library loaded before torch", flush=True)
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT, out], capture_output=True, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    rng = np.random.default_rng(3)
    q = torch.from_numpy(rng.standard_normal((300, 24)).astype(np.float16)).cuda()
    k = torch.from_numpy(rng.standard_normal((500, 24)).astype(np.float16)).cuda()
    v = torch.from_numpy(rng.standard_normal((500, 5)).astype(np.float32)).cuda()
    s = gs.gauss_sum_fwd(q, k, v, 0.05)
    torch.cuda.synchronize()
    assert np.array_equal(np.load(out), s.cpu().numpy())
