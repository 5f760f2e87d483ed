"""Converts a synthetic block into the plain arrays the CPU oracle takes."""
import numpy as np

import oracle
from synth import PSI_FIELDS, bf16_bits


def psi_f64(block):
    return {k: oracle.bf16_to_f64(bf16_bits(block.psi[k])) for k in PSI_FIELDS}


def oracle_inputs(block):
    """Host copies of every input, bf16 tables kept as bit patterns."""
    return dict(
        H=oracle.bf16_to_f64(bf16_bits(block.H)),
        H_bits=bf16_bits(block.H),
        W_bits=bf16_bits(block.W),
        E_bits=bf16_bits(block.E),
        h_c=oracle.bf16_to_f64(bf16_bits(block.h_c)),
        x0=block.x0.cpu().numpy().astype(np.int64),
        verifier=block.verifier.cpu().numpy(),
        psi=psi_f64(block),
        alpha=block.alpha,
        b_g=block.b_g,
    )


def f64_to_bf16_bits(x):
    """Bits of values that are exactly representable in bf16 (asserted)."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not representable in bf16"
    return (u >> 16).astype(np.uint16)
