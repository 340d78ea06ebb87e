"""Oracle for the AR-DiT chunk-denoise block -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy implementation of what one AR-DiT transformer
block computes for one chunk of latent tokens in one denoising step.  It is
written from the definition of the block (see ``ardit_ref``) and shares no
code with the HIP library: only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  The product path
never calls it.

Parity status per function (what pins it is listed in each docstring):
every function here is pinned by a CPU test against a closed form, an
invariant the paper fixes, or a brute-force loop on tiny inputs, except the
numerics of a trained model, which no printed value pins ("parity unpinned":
the paper prints no worked example of the block).
"""
from .ardit_ref import (  # noqa: F401
    DTYPE, timestep_sinusoid, silu, linear, rms_norm, gelu_tanh, rope_split,
    rope_inv_freq, chunk_positions, rope3d, attention, time_modulation,
    context_kv, block_forward, full_sequence_forward,
)
from . import sparse_ref  # noqa: F401
from . import fp8_ref  # noqa: F401
from . import chunk_ref  # noqa: F401
from . import control_ref  # noqa: F401
