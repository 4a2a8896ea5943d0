"""Oracle: a plain, slow, CPU-only NumPy implementation of the stream-batched
rectified-flow step.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the bench's CPU
baseline leg may import this package. The product path (the HIP library and its
Python binding) never calls it, and it shares no code with that path: it has its
own blob reader and its own arithmetic. Its inputs come from `workloads`, which
holds no arithmetic of the method.

What it computes (StreamFlow, arXiv 2511.22009):
  * the velocity-network forward v = F(x_k, t_k) over a batch of in-flight latents,
    each at its own timestep (Sec. 3.2, Eq. 5), looping one sample at a time so the
    batch result is exactly each sample run alone;
  * the per-sample Euler update x' = x + dt * v with dt = t_next - t
    (Sec. 3.1.1 discretization; Alg. 1, its final update);
  * the queue shift: new noise enters slot 0, every latent moves one slot on, and the
    oldest leaves once the pipeline is full (Sec. 3.4.1-3.4.2; Alg. 2);
  * the whole Alg. 2 driver over M images;
  * PeRFlow's time-window conversion of a noise prediction into a velocity, batched
    over heterogeneous timesteps (Sec. 2 time windows; Sec. 3.3; Alg. 1), in
    `oracle.perflow`.

The network itself is not in the paper (the paper runs a pretrained UNet that
predicts noise); this oracle uses a DiT-style adaLN transformer that outputs v
directly, with every reading of an unstated detail fixed in the module docstrings.

Precision: fp32 by default (`dtype=np.float64` runs the same steps in fp64 as a
self-check). Parity status per function is stated in each docstring; the full
network output has no external value to compare against ("parity unpinned"
against outside numbers) and is pinned by brute force, closed forms and the
method's invariants in the tests.
"""
from .weights import OracleModel, load_blob
from .dit import (timestep_frequencies, timestep_embedding, modulation_table, patchify,
                  unpatchify, layer_norm, gelu_tanh, silu, attention, residual_one, forward_one,
                  velocity)
from .stream import euler, stream_step, run_stream, sequential_sample, noise_latent
from . import perflow

__all__ = [
    "OracleModel", "load_blob", "timestep_frequencies", "timestep_embedding",
    "modulation_table", "patchify", "unpatchify", "layer_norm", "gelu_tanh", "silu",
    "attention", "residual_one", "forward_one", "velocity", "euler", "stream_step", "run_stream",
    "sequential_sample", "noise_latent", "perflow",
]
