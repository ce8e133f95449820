"""One Muon step on seeded inputs through the C ABI, reduced to a digest of
the resulting parameter and momentum bits.  The serialised-launch test runs
it in-process and, as `python -m tests.gpu_child_step`, in a child process
with every kernel launch serialised; the digests must be equal."""
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# chunks of few tiles: they alternate between the caller's stream and the
# handle's second one
SHAPES = [(512, 1024)] * 3 + [(768, 768)] + [(256, 256)] * 2 + [(200, 300)]


def run(shapes=SHAPES, key=31):
    import numpy as np
    import torch

    from paper_2609_21594_amd import synth
    from paper_2609_21594_amd.binding import Muon

    def rng(*k):
        return np.random.Generator(np.random.PCG64(np.random.SeedSequence([key, *k])))

    def bf(a):
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()

    W = [bf(synth.draw(s, 0.02, "bf16", rng(i, 0))) for i, s in enumerate(shapes)]
    G = [bf(synth.draw(s, 1e-3, "bf16", rng(i, 1))) for i, s in enumerate(shapes)]
    M = [torch.from_numpy(synth.draw(s, 1e-3, "f32", rng(i, 2))).cuda() for i, s in enumerate(shapes)]
    torch.cuda.synchronize()
    m = Muon(0)
    try:
        m.step(W, G, M, lr=0.02, beta=0.95, weight_decay=0.01, ns_precision="bf16")
        torch.cuda.synchronize()
    finally:
        m.close()
    h = hashlib.sha256()
    for t in W + M:
        h.update(t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy().tobytes())
    return h.hexdigest()


if __name__ == "__main__":
    print(json.dumps(run()), flush=True)
