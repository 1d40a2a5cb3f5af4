"""dv_encode_noalloc (workspace in the library's static scratch array, for callers that cannot
allocate) against dv_encode (the handle's workspace) through the C ABI: two calls in a row, the second smaller, equal bit for
bit (results do not depend on the internal batch size, and the no-allocation entry point cuts
batches to what its array holds), in gate mode, with reuse off and with every token reused."""
import numpy as np
import pytest

import synth
from paper_2506_14107_amd import dejavu as dj

from .gpu_util import dev, encoder, host, require_gpu

pytestmark = pytest.mark.gpu


def _both(torch, enc, fr, G, tau):
    n = fr.shape[0]
    m = enc.model
    want_e, want_m, _ = enc.encode(fr, G, tau)
    got_e = torch.empty((n, m.width), dtype=torch.float32, device="cuda")
    got_m = torch.empty((n, m.depth, m.n_tokens), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    enc.encode_noalloc(fr, G, tau, got_e, got_m)
    torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info()[0]
    return host(want_e), host(want_m), host(got_e), host(got_m), free0 - free1


@pytest.mark.parametrize("name,batch,calls,G", [
    ("tiny", 8, (8, 5), 4),          # fp32 model: the array holds the handle's whole batch
    ("vit_l14", 64, (40, 13), 8),    # bf16: the array holds 16 frames, the handle 64
])
def test_noalloc_equals_encode(name, batch, calls, G):
    torch = require_gpu()
    w = synth.get_config(name)
    m = w.model
    blob = synth.make_blob(m, w.weight_seed)
    enc = encoder(m, blob, batch)
    fr_all = synth.render_frames(w.video, m.image_size, 0, max(calls))
    taus = [float(np.float32(w.tau if w.tau is not None else 0.9)), float("-inf"), float("inf")]
    for k, n in enumerate(calls):
        fr = dev(fr_all[:n])
        for tau in taus:
            print(f"[noalloc {name}] call {k}: {n} frames, G {G}, tau {tau}", flush=True)
            we, wm, ge, gm, grew = _both(torch, enc, fr, G, tau)
            assert np.array_equal(ge, we), f"embeddings differ from dv_encode (tau {tau})"
            assert np.array_equal(gm, wm), f"reuse maps differ from dv_encode (tau {tau})"
            if k > 0:
                assert grew == 0, f"device memory in use grew by {grew} bytes during the call"
            if np.isfinite(tau):
                rho = float((wm[[f for f in range(n) if f % G]] != 0).mean())
                print(f"[noalloc {name}] reuse {rho:.3f}", flush=True)
    enc.close()


def test_noalloc_rejects_a_group_larger_than_the_array():
    torch = require_gpu()
    w = synth.get_config("vit_l14")
    m = w.model
    enc = encoder(m, synth.make_blob(m, w.weight_seed), 32)
    fr = dev(synth.render_frames(w.video, m.image_size, 0, 24))
    e = torch.empty((24, m.width), dtype=torch.float32, device="cuda")
    with pytest.raises(dj.DejaVuError) as err:   # one group of 24 ViT-L/14 frames: ~174 MB
        enc.encode_noalloc(fr, 24, 0.9, e)
    assert err.value.code == dj.DV_ENOMEM and "scratch" in dj.dv_last_error()
    enc.close()
