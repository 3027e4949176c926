"""The binding loaded before torch has touched the device.

The torch wheel ships its own HIP runtime under the system runtime's soname;
the library must end up on the same runtime as the tensors it is given
whichever is imported first.  The order can only be set up in a fresh
interpreter, so one child process runs it: the binding's lib() first, then
a torch tensor, then a launch through the C ABI."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
sys.path.insert(0, {root!r})
from paper_2606_26472_amd import epikv as E
E.lib()
import torch
cfg = E.default_cfg(batch=3)
st = torch.full((E.state_bytes(cfg),), 0x55, dtype=torch.uint8, device="cuda")
E.epikv_state_init(cfg, st)
torch.cuda.synchronize()
assert int(st.count_nonzero()) == 0          # every byte reset
print("launch after binding-first load: ok", flush=True)
"""


def test_binding_loaded_before_torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = subprocess.run([sys.executable, "-c", CHILD.format(root=ROOT)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "ok" in r.stdout
