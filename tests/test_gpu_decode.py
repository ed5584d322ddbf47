"""GPU parity of the greedy decode loop (Algorithm 1) around the spliced
attention: paper_2605_30574_amd.decode on the GPU (this library's kernel for
each layer's KV append and attention) against oracle.decoder (float64 on
the CPU), teacher-forced -- both decode the GPU's tokens, so a near tie
cannot send the two down different trajectories.

Bars (tiny float32 model; only q, k, v and the caches are bf16 on both
sides), derived on the CPU in tests/decode_bar.py from the attention bar
alone -- twice what the reference decoder shows when every attention output
is moved by 1e-3 on average (independent noise, or one coherent relative
error per call):
  * logits of every active cell within LOGIT_REL of the oracle's, relative
    to max(1, largest logit magnitude);
  * appended cache rows at layer 0 (a function of the embeddings alone)
    within one bf16 rounding of the float32-vs-float64 projections; at
    layers >= 1 each element within ROW_REL of the layer's row rms, and at
    most a ROW_FLIP_FRAC fraction of the elements with other bits.
A wiring mistake (a wrong position, layer, splice or cache row) moves logits
by tens of percent.  The argmax must be equal wherever the oracle's top two
logits are more than twice the bar apart; cells stop at EOS on both sides
alike (the EOS id is taken from the first pass, so some cells do stop and
are skipped from then on)."""
import numpy as np
import pytest
import torch

import decode_bar
import gpu_common as gc
import paper_2605_30574_amd as sp
from oracle import decoder as ref
from paper_2605_30574_amd import decode
import workloads
from workloads.model import make_weights

pytestmark = pytest.mark.gpu

# derived by decode_bar.derive() (test_decode_bar.py checks they still are)
LOGIT_REL = 0.008
ROW_REL = 0.033
ROW_FLIP_FRAC = 0.83


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sp.load_library()


@pytest.mark.parametrize("name", decode_bar.CASES)
def test_decode_loop_matches_oracle(name):
    w = decode_bar.case(name)
    m = decode_bar.MODEL
    lw = workloads.cell_lw(w)
    C = lw.shape[0]
    wt_cpu = make_weights(w, m, dtype=torch.float32)
    wt_gpu = {"embed": wt_cpu["embed"].cuda(), "lm_head": wt_cpu["lm_head"].cuda(), "norm_f": wt_cpu["norm_f"].cuda(),
              "layers": [{k: v.cuda() for k, v in L.items()} for L in wt_cpu["layers"]]}
    caches = [gc.gpu_layer(w, l, n_cells=C) for l in range(w.n_layers)]
    prompts = [{k: v for k, v in gc.host(c).items() if k in ("clean_k", "clean_v", "donor_k", "donor_v")} for c in caches]
    gpu = decode.SweepDecoder(w, m, wt_gpu, caches, lw)
    cpu = ref.ReferenceDecoder(w, m, decode_bar.f64_weights(wt_cpu), prompts, lw)
    steps = np.zeros(C, dtype=np.int32)
    tokens = np.full(C, 11, dtype=np.int64)   # the token after prefill: the same for every cell
    eos = None   # chosen after the first pass (the token cell 2 emits), so some cells do stop
    stopped, worst = 0, 0.0
    for it in range(w.n_steps):
        if (steps < 0).all():
            break
        gc.announce(f"decode {name} pass {it} steps={steps.tolist()}")
        nxt, logits = gpu.step(torch.as_tensor(tokens, device="cuda"), steps)
        torch.cuda.synchronize()
        g = logits.cpu().numpy().astype(np.float64)
        r = cpu.forward(tokens, steps)
        act = steps >= 0
        scale = max(1.0, float(np.abs(r[act]).max()))
        err = float(np.abs(g[act] - r[act]).max()) / scale
        worst = max(worst, err)
        assert err <= LOGIT_REL, f"{name} pass {it}: logits rel err {err:.2e}"
        top2 = np.sort(r[act], axis=-1)[:, -2:]
        clear = (top2[:, 1] - top2[:, 0]) > 2 * LOGIT_REL * scale
        gn = nxt.cpu().numpy()
        assert np.array_equal(gn[act][clear], ref.greedy(r[act])[clear]), f"{name} pass {it}: argmax"
        if eos is None:
            eos = int(gn[2])
        new_steps = decode.advance(steps, gn, eos, w.n_steps)
        stopped += int(((new_steps < 0) & act & (gn == eos)).sum())
        tokens = np.where(new_steps >= 0, gn, tokens)
        steps = new_steps
    gc.announce(f"decode {name}: worst logits rel err {worst:.2e} over {it + 1} passes")
    assert stopped >= 1, f"{name}: no cell reached EOS"
    # the rows the GPU appended are the rows the reference stored: at layer 0
    # (a function of the embeddings alone) to within one bf16 rounding of the
    # float32-vs-float64 projections, deeper element by element to within the
    # derived bars
    for l in range(w.n_layers):
        for kind, mine in (("gen_k", cpu.gen_k[l]), ("gen_v", cpu.gen_v[l])):
            got_bits = workloads.to_numpy(caches[l][kind])
            written = mine != 0
            if l == 0:
                got, want = ref.from_bf16_bits(got_bits), ref.from_bf16_bits(mine)
                assert np.allclose(got[written], want[written], rtol=2 ** -7, atol=1e-6), f"{name} layer 0: {kind}"
            else:
                dev, flip = decode_bar.row_deviation(mine, np.where(written, got_bits, 0).astype(np.uint16))
                gc.announce(f"decode {name} layer {l} {kind}: deviation {dev:.2e} of rms, {flip:.3f} flipped")
                assert dev <= ROW_REL, f"{name} layer {l}: {kind} deviation {dev:.2e} of the rows' rms"
                assert flip <= ROW_FLIP_FRAC, f"{name} layer {l}: {kind} {flip:.3f} of the elements differ"
