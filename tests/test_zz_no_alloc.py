"""The allocation-free forward (sats_mlp_forward_noalloc) against
sats_mlp_forward: the same kernels on the library's fixed scratch array, so
the outputs must agree bit for bit -- on two calls in a row, the second with
a smaller input, so that the second call runs over the first call's leftovers
in the shared array."""
import sys

import numpy as np
import pytest

from harness import to_dev, from_dev, weights_dev
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2607_08991_amd as sats
    sats.load()


def _both(c, ts, lut):
    """Output of sats_mlp_forward and of sats_mlp_forward_noalloc on the same inputs."""
    import torch
    import paper_2607_08991_amd as sats
    x = to_dev(c["x"], "bf16")
    n, d = c["x"].shape
    L, _, dff = c["W_gate"].shape
    w = list(weights_dev(c, "bf16"))
    ids = to_dev(np.asarray(c["token_ids"], np.int32), "bf16") if lut is not None else None
    dl = to_dev(lut, "bf16") if lut is not None else None
    thr = torch.tensor(np.asarray(ts, np.float32)).cuda()
    ref = torch.empty((n, d), dtype=torch.bfloat16, device="cuda")
    got = torch.full((n, d), 7.0, dtype=torch.bfloat16, device="cuda")
    sats.sats_mlp_forward(x, ids, *w, thr, dl, ref, n, d, dff, L)
    sats.sats_mlp_forward_noalloc(x, ids, *w, thr, dl, got, n, d, dff, L)
    torch.cuda.synchronize()
    sats.sats_device_status()
    return from_dev(ref), from_dev(got)


def test_noalloc_matches_forward_on_two_calls_the_second_smaller():
    from oracle import calibrate
    cfg = get_config("c2_llama8b_layer_bf16")
    wg, wu, wd = synth.layer_weights(cfg.seed, 0, cfg.d, cfg.d_ff, cfg.dtype)
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "thresholds.json")))
    ts = np.asarray(g[cfg.name]["thresholds"], np.float32)
    big = dict(x=synth.decode_x(cfg, 1), token_ids=np.zeros(1, np.int32), W_gate=wg[None], W_up_T=wu[None],
               W_down=wd[None])
    small = synth.small_case(81, 2, 256, 1000, "bf16", 1, vocab=40, n_dense_ids=12, w_std=1 / 16)
    xcal = synth.activations(981, synth.S_CAL, 24, 256, "bf16")
    ts_small = calibrate.calibrate_stack(xcal, small["W_gate"], small["W_up_T"], small["W_down"], [0.5, 0.5], "bf16")
    batch = synth.small_case(82, 2, 256, 1024, "bf16", 4, vocab=40, n_dense_ids=12, w_std=1 / 16)
    xcal = synth.activations(982, synth.S_CAL, 24, 256, "bf16")
    ts_batch = calibrate.calibrate_stack(xcal, batch["W_gate"], batch["W_up_T"], batch["W_down"], [0.5, 0.5], "bf16")
    # the Llama layer (single token), then a smaller two-layer stack with a base-path and a sparse-path token,
    # then a 4-token batch, then the Llama layer again
    runs = [("llama layer, 1 token", big, ts, None)]
    for tok in (int(np.argmax(small["route_lut"])), int(np.argmin(small["route_lut"]))):
        runs.append((f"256 x 1000 stack, id {tok}", dict(small, token_ids=np.array([tok], np.int32)), ts_small,
                     small["route_lut"]))
    runs.append(("256 x 1024 stack, 4 tokens", batch, ts_batch, batch["route_lut"]))
    runs.append(("llama layer again", big, ts, None))
    for name, c, t, lut in runs:
        ref, got = _both(c, t, lut)
        say(f"{name}: equal {np.array_equal(ref, got)}")
        np.testing.assert_array_equal(ref, got)


def test_noalloc_rejects_a_call_past_its_scratch():
    import torch
    import paper_2607_08991_amd as sats
    n, d, dff = 64, 4096, 14336   # 64 tokens at the Llama shape need far more than 16 MiB
    x = torch.zeros((n, d), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((d * dff,), dtype=torch.bfloat16, device="cuda")
    thr = torch.zeros(1, device="cuda")
    with pytest.raises(sats.SatsError) as e:
        sats.sats_mlp_forward_noalloc(x, None, w, w, w, thr, None, x, n, d, dff, 1)
    assert e.value.code == -4 and "allocation-free" in str(e.value)
