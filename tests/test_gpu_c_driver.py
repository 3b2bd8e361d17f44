"""The partition driven through its C ABI alone, from a C++ program with no
Python or torch in its process (tests/host/abi_driver.cpp, linked against
libgp.so by the build): device buffers from hipMalloc, M forwards, M
re-materialising backwards in reverse micro-batch order, one update
(Sections 2.2-2.3).  Its boundary outputs, accumulated gradients and updated
parameters are compared with the fp64 oracle's GPipe step on the same seeded
inputs (fp32: max-abs relative error <= 1e-4 per tensor).
"""
import os
import struct
import subprocess

import numpy as np
import pytest

import synth
from oracle import gpipe
from parity import compare_grads, rel_err

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "host", "_bin", "abi_driver")
CFG = synth.CONFIGS["tiny"].with_(name="tiny_boundary_c", loss="none")


def _param_ids():
    # the C ABI's parameter numbering (include/gp.h), encoder layers only
    from paper_1811_06965_amd.gp import PARAM_ID
    return PARAM_ID


@pytest.mark.parametrize("micro", [1, 4])
def test_c_program_runs_a_gpipe_step_that_matches_the_oracle(tmp_path, micro):
    if not os.path.exists(DRIVER):
        raise FileNotFoundError(f"{DRIVER} is missing: run the build (python -m paper_1811_06965_amd.build)")
    cfg = CFG.with_(micro=micro)
    case = synth.make_case(cfg, 31, perturb=True)
    lr = 1e-3
    ref = gpipe.gpipe_step(cfg, case, cfg.micro, lr=lr)
    ids = _param_ids()
    recs = [(l, name, np.ascontiguousarray(arr, dtype=np.float32))
            for l, p in enumerate(case["layers"]) for name, arr in p.items()]
    n = cfg.batch // cfg.micro
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(inp, "wb") as f:
        f.write(struct.pack("<8i", cfg.layers, cfg.d_model, cfg.d_ff, cfg.heads, cfg.seq, n, cfg.micro, len(recs)))
        f.write(struct.pack("<2f", cfg.ln_eps, lr))
        for l, name, a in recs:
            f.write(struct.pack("<iiq", l, ids[name], a.size))
            f.write(a.tobytes())
        f.write(np.ascontiguousarray(case["x"], dtype=np.float32).tobytes())
        f.write(np.ascontiguousarray(case["dy"], dtype=np.float32).tobytes())
    print("abi_driver", cfg.name, "M =", cfg.micro, flush=True)
    r = subprocess.run([DRIVER, str(inp), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    got = np.fromfile(out, dtype=np.float32)
    N, S, D = cfg.batch, cfg.seq, cfg.d_model
    off = 0

    def take(shape):
        nonlocal off
        k = int(np.prod(shape))
        a = got[off:off + k].reshape(shape)
        off += k
        return a

    y, dx = take((N, S, D)), take((N, S, D))
    grads = [dict() for _ in range(cfg.layers)]
    for l, name, a in recs:
        grads[l][name] = take(a.shape)
    params = [dict() for _ in range(cfg.layers)]
    for l, name, a in recs:
        params[l][name] = take(a.shape)
    assert off == got.size
    assert rel_err(y, ref["y"]) <= 1e-4
    assert rel_err(dx, ref["dx"]) <= 1e-4
    compare_grads(grads, {}, ref["grads"], {}, "rel", 1e-4)
    for l, name, _ in recs:
        assert rel_err(params[l][name], ref["layers"][l][name]) <= 1e-6, (l, name)
