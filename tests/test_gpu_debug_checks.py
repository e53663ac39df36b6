"""The library's debug mode (ESTP_DEBUG_CHECKS=1): cu_seqlens is checked on the host before any
kernel reads it, and the device-built lists of live 256-row blocks (importance) and live chunks
(pooling) are compared with their definitions before the kernels that use them run.

The mode is read once per process, so it runs in a child process.  The child first confirms that
the mode is on (and stops otherwise, before any malformed input is passed), then:
* runs ragged batches that take both work lists and writes the results for the parent, which
  compares them bit for bit with its own run in the normal mode;
* passes malformed cu_seqlens arrays (which the normal mode does not inspect) and expects every
  one to be refused on the host with ESTP_ERR_INVALID_ARG.
"""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import paper_2608_15592_amd as estp

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# one prompt over 8192 tokens sends the pooling through its list of live chunks
LENGTHS = [9000] + [1000, 10, 5, 300, 2, 700, 1, 40, 257, 256, 3, 999] * 3
MAX_LEN = max(LENGTHS)

CHILD = r"""
import sys, numpy as np, torch
sys.path.insert(0, ROOT)
import paper_2608_15592_amd as estp
from paper_2608_15592_amd import _lib
from tests.test_gpu_debug_checks import MAX_LEN, make_inputs, run_calls
lib = estp.load()
if lib.estp_debug_checks() != 1:
    print("debug checks are off"); sys.exit(3)
inp = make_inputs()
np.savez(OUT, **run_calls(inp))
# malformed cu_seqlens: refused on the host before any kernel
Q, K, X, S, H = inp["Q"], inp["K"], inp["X"], inp["S"], inp["H"]
n = X.shape[0]
good = inp["cu"].cpu().numpy()
bad = {
    "nonzero first offset": np.concatenate([[1], good[1:]]),
    "empty prompt": np.concatenate([good[:3], [good[2]], good[4:]]),
    "decreasing": np.concatenate([good[:5], [good[4] - 1], good[6:]]),
    "last offset past n_tok": np.concatenate([good[:-1], [n + 5]]),
}
for name, cu in bad.items():
    cud = torch.tensor(cu, dtype=torch.int32, device="cuda")
    for call in ("importance", "pool", "misalignment"):
        try:
            if call == "importance":
                estp.attn_importance(Q, K, cud, MAX_LEN)
            elif call == "pool":
                estp.combine_pool(X, S, H, cud, MAX_LEN, 0.5, 0.5)
            else:
                if name == "last offset past n_tok":
                    continue  # the call does not state n_tok
                estp.misalignment(H, S, cud)
        except estp.EstpError as e:
            assert e.status == 1 and "debug check" in str(e), (name, call, str(e))
            print(f"refused ({call}, {name}): {e}")
            continue
        print(f"NOT refused: {call}, {name}"); sys.exit(4)
# a prompt longer than the stated max_seqlen
try:
    estp.attn_importance(Q, K, inp["cu"], MAX_LEN - 1)
    print("NOT refused: max_seqlen"); sys.exit(4)
except estp.EstpError as e:
    assert e.status == 1 and "debug check" in str(e)
torch.cuda.synchronize()
print("child ok")
"""


def make_inputs():
    g = torch.Generator(device="cuda").manual_seed(21)
    n = sum(LENGTHS)
    cu = torch.tensor(np.concatenate([[0], np.cumsum(LENGTHS)]), dtype=torch.int32, device="cuda")
    Q = torch.randn(1, n, 8, 64, device="cuda", generator=g).to(torch.bfloat16)
    K = torch.randn(1, n, 2, 64, device="cuda", generator=g).to(torch.bfloat16)
    X = torch.randn(n, 512, device="cuda", generator=g).to(torch.bfloat16)
    H = torch.rand(n, device="cuda", generator=g) * 5
    S = torch.rand(n, device="cuda", generator=g) * 1e-3
    return {"Q": Q, "K": K, "X": X, "H": H, "S": S, "cu": cu}


def run_calls(inp):
    S = estp.attn_importance(inp["Q"], inp["K"], inp["cu"], MAX_LEN)
    pooled, e, top = estp.combine_pool(inp["X"], inp["S"], inp["H"], inp["cu"], MAX_LEN, 0.5, 0.5, 1.0, "zscore")
    counts = estp.misalignment(inp["H"], inp["S"], inp["cu"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in (("S", S), ("pooled", pooled), ("e", e), ("top", top), ("counts", counts))}


def test_debug_checks_pass_valid_batches_and_refuse_malformed_offsets(tmp_path):
    lib = estp.load()
    assert lib.estp_debug_checks() == 0  # this process: normal mode
    ref = run_calls(make_inputs())
    out = str(tmp_path / "debug_run.npz")
    env = dict(os.environ, ESTP_DEBUG_CHECKS="1")
    code = CHILD.replace("ROOT", repr(ROOT)).replace("OUT", repr(out))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    print(r.stdout[-4000:])
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "child ok" in r.stdout
    got = np.load(out)
    for k in ref:
        np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
