"""GPU parity of the HIP partition against the fp64 oracle (through the C ABI).

Tolerances: fp32 partitions, max-abs relative error <= 1e-4 on outputs,
input gradients, loss, every parameter gradient and the updated parameters;
bf16 partitions, <= 2e-2 on outputs, input gradients and loss, and cosine
similarity >= 0.999 per parameter-gradient tensor.
"""
import numpy as np
import pytest

import synth
from parity import compare_grads, rel_err, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _run(cfg, seed, perturb=True, M=None, lr=0.0):
    from oracle import gpipe
    from paper_1811_06965_amd.runtime import Partition
    case = synth.make_case(cfg, seed, perturb=perturb)
    M = cfg.micro if M is None else M
    ref = gpipe.gpipe_step(cfg, case, M, lr=lr)
    with Partition(cfg, micro=M) as part:
        part.load_params(case["layers"], case["head"])
        inp = part.device_inputs(case)
        out = part.step(inp["x"], inp["mem"], inp["dy"], lr=0.0)
        torch.cuda.synchronize()
        gl, gh = part.grads()
        res = dict(y=to_np(out["y"]), dx=to_np(out["dx"]), loss=out["loss"],
                   dmem=None if out["dmem"] is None else to_np(out["dmem"]), grads=(gl, gh))
    return case, ref, res


def _check(cfg, ref, res, out_tol, grad_mode, grad_tol):
    assert rel_err(res["y"], ref["y"]) <= out_tol, rel_err(res["y"], ref["y"])
    assert rel_err(res["dx"], ref["dx"]) <= out_tol, rel_err(res["dx"], ref["dx"])
    if cfg.loss != "none":
        assert abs(res["loss"] - ref["loss"]) <= out_tol * abs(ref["loss"]), (res["loss"], ref["loss"])
    if cfg.kind == "decoder":
        assert rel_err(res["dmem"], ref["dmem"]) <= out_tol
    gl, gh = res["grads"]
    compare_grads(gl, gh, ref["grads"], ref["head_grads"], grad_mode, grad_tol)


TINY = synth.CONFIGS["tiny"]


@pytest.mark.parametrize("seed", [0, 1])
def test_tiny_fp32_matches_oracle(seed):
    case, ref, res = _run(TINY, seed)
    _check(TINY, ref, res, 1e-4, "rel", 1e-4)


def test_tiny_fp32_config_init_matches_oracle():
    """The workload's own initialisation (biases 0, LayerNorm gain 1)."""
    case, ref, res = _run(TINY, 2, perturb=False)
    _check(TINY, ref, res, 1e-4, "rel", 1e-4)
