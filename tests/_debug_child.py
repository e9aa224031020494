"""Child process of tests/test_gpu_debug_build.py: runs the cases of that test
through the library named on the command line and saves every output.  Not a
test module (pytest does not collect it)."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def run_cases():
    """(name -> array) of the outputs of the cases, through whatever library
    paper_2608_23167_amd._lib has loaded."""
    import torch
    from synthetic import WORKLOADS, initial_tokens, make_weights, mid_generation_state
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    out = {}
    dev = "cuda:0"

    def load(dec, state, step):
        t, pi, pw, ps = state
        dec.tokens.copy_(torch.from_numpy(np.asarray(t, np.int32)).to(dev))
        dec.pred_ids.copy_(torch.from_numpy(np.asarray(pi, np.int32)).to(dev))
        dec.pred_w.copy_(torch.from_numpy(np.asarray(pw, np.float32)).to(dev))
        dec.pred_step.copy_(torch.from_numpy(np.asarray(ps, np.int32)).to(dev))
        dec.step_idx = step

    # tiny float32: a free-running generation of two blocks
    wl = WORKLOADS["tiny"]
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1).to(dev)
    dec = Decoder(wl, DeviceModel(wl.model, mw))
    dec.generate(initial_tokens(wl).to(dev), max_steps=2 * wl.steps_per_block())
    torch.cuda.synchronize()
    out["tiny_tokens"] = dec.tokens.cpu().numpy()
    out["tiny_pred_w"] = dec.pred_w.cpu().numpy()
    # LLaDA-8B shape, two layers, bfloat16: block start and cached step, and a
    # batch of three prompts of different lengths
    for name, batch, lens in (("llada_gen256", 1, None), ("llada_gen256", 3, [256, 200, 131])):
        wl = WORKLOADS[name].replace(batch=batch)
        wl = wl.replace(model=wl.model.with_layers(2))
        mw = make_weights(wl.model, seed=0, norm_jitter=0.1).to(dev)
        dec = Decoder(wl, DeviceModel(wl.model, mw), prompt_lens=lens)
        state = mid_generation_state(wl, 1, 1, seed=3)
        for first in (True, False):
            load(dec, state, 1)
            logits = torch.empty(batch * dec.max_rows * wl.model.vocab, device=dev)
            info = dec.step(1, first, logits=logits)
            torch.cuda.synchronize()
            tag = f"{name}_b{batch}_{'start' if first else 'cached'}"
            out[tag + "_logits"] = logits[: batch * info.n_out * wl.model.vocab].cpu().numpy()
            out[tag + "_tokens"] = dec.tokens.cpu().numpy()
            out[tag + "_pred_ids"] = dec.pred_ids.cpu().numpy()
    return out


if __name__ == "__main__":
    from paper_2608_23167_amd import _lib
    _lib.use_library(sys.argv[1])
    np.savez(sys.argv[2], **run_cases())
