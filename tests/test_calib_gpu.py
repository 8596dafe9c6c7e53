"""GPU parity of the calibration kernels (masq_channel_range,
masq_smoothing_factors, masq_quantize_weight) against the oracle's
definitions (oracle/calibration.py): bit-exact, through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from oracle import calibration as cal
from oracle.bf16 import bf16_round

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    assert torch.cuda.is_available(), "GPU tests need an MI355X visible to torch"
    from paper_2603_04800_amd import ops as o
    return o


def _check(ops, x, mod, w, n_mod, act, bits=(8, 4)):
    dev = torch.device("cuda:0")
    xt = torch.from_numpy(x).to(dev, torch.bfloat16 if act == "bf16" else torch.float32)
    mt = torch.from_numpy(np.asarray(mod, np.int32)).to(dev)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(dev)
    rng = ops.channel_range(xt, mt, n_mod)
    s, inv = ops.smoothing_factors(rng, wt)
    torch.cuda.synchronize()
    wmax = cal.weight_range(w)
    s_text_ref = None
    for m in range(n_mod):
        r_ref = cal.channel_range(x, mod, m)
        assert np.array_equal(rng[m].cpu().numpy(), r_ref.astype(np.float32)), f"range {m}"
        s_ref, inv_ref = cal.smoothing_factor(r_ref, wmax)
        assert np.array_equal(s[m].cpu().numpy().view(np.uint32), s_ref.view(np.uint32)), f"s {m}"
        assert np.array_equal(inv[m].cpu().numpy().view(np.uint32), inv_ref.view(np.uint32))
        if m == 0:
            s_text_ref = s_ref
    for b in bits:
        # each side quantises with its own text factor (equal bit for bit above)
        wq, ws = ops.quantize_weight(wt, s[0].contiguous(), bits=b)
        torch.cuda.synchronize()
        wq_ref, ws_ref, _ = cal.quantize_weight(w, s_text_ref, b)
        assert np.array_equal(wq.cpu().numpy(), wq_ref), f"{b}-bit codes"
        assert np.array_equal(ws.cpu().numpy().view(np.uint32), ws_ref.view(np.uint32))


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_small_calibration_with_invalid_ids_and_empty_modality(ops, act):
    rng = np.random.default_rng(3)
    T, K, N = 300, 96, 80
    mod = rng.integers(0, 3, T).astype(np.int32)          # modality 3 of 4 has no tokens
    mod[[5, 77, 200]] = [7, -1, 4]                          # ids outside [0, 4): no modality
    x = (rng.standard_normal((T, K)) * rng.uniform(0.1, 30, K)).astype(np.float32)
    x[:, 3] = 0.0                                           # an all-zero channel (floored)
    if act == "bf16":
        x = bf16_round(x)
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    w[:, 5] = 0.0                                           # an all-zero output channel
    _check(ops, x, mod, w, 4, act)


def test_prefill_workload_calibration(ops):
    """The 4096-token prefill layer's X and the 3584 x 18944 float weight."""
    cfg = synth.CONFIGS[1]
    li = synth.make_layer_inputs(cfg, 0)
    p = cfg.projections[0]
    _check(ops, li.x[p.input_key], li.modality, li.w[p.name], cfg.n_mod, cfg.act_dtype,
           bits=(8,))


@pytest.mark.parametrize("cfg_index,bits", [(0, 8), (3, 8), (1, 4)])
def test_gpu_assisted_layer_calibration_equals_host(ops, cfg_index, bits):
    """calibrate_layer_gpu (ranges, factors and Q(S_t W) on the GPU) gives the
    host calibration's artifacts array for array, the compensation factors
    included."""
    from paper_2603_04800_amd import calibrate
    cfg = synth.CONFIGS[cfg_index]
    li = synth.make_layer_inputs(cfg, 0)
    p = cfg.projections[0]
    x, w = li.x[p.input_key], li.w[p.name]
    host = calibrate.calibrate_layer(x, li.modality, w, cfg.n_mod, cfg.rank, cfg.lr_dtype,
                                     weight_bits=bits)
    gpu = calibrate.calibrate_layer_gpu(x, li.modality, w, cfg.n_mod, cfg.rank, cfg.lr_dtype,
                                        weight_bits=bits)
    for k in ("inv_smooth", "s32", "wq", "w_scale", "l_down", "r_up"):
        assert np.array_equal(np.asarray(gpu[k]), np.asarray(host[k])), k
