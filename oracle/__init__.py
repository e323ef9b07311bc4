"""Oracle for the integrated fixed-point quantized convolution (IFQ-Net).

TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
baseline may import this package. It is a plain, slow CPU implementation of
what the GPU path computes, written from the paper and sharing no code with
the GPU library:

  ifq_oracle.c   integer conv (int64 accumulation), fp64 threshold fold,
                 integer codes, max-pool on codes, residual join (C, OpenMP)
  core.py        ctypes wrappers over ifq_oracle.c
  stack.py       walks a synthetic layer stack through the C oracle (O_int)
  float_chain.py the defining float chain conv -> BN -> quantizer in fp64
                 (O_float), used as the invariant the integer path must meet
  brute.py       pure-Python loops for tiny layers
  layout.py      the 2-bit packed code layout (4 codes per byte along C)

Parity status per function (what pins it is in the tests):
  conv acc       pinned: brute force, float64 conv2d of integer tensors,
                 closed forms
  fold + codes   pinned: exhaustive check over every reachable sum against the
                 float chain, the float-chain invariant on stack layers, a
                 mutation test of the sign flip
  max-pool       pinned: brute force, commutation with a monotone code map
  2-bit layout   pinned: round trip, the paper's feature-map size arithmetic
  residual join  parity unpinned: the paper has no residual networks; pinned
                 only by its own definition against the float chain
"""
from .core import (conv_acc, fold, codes, maxpool, join_coeffs, join_codes,
                   num_threads, MUTATE_NO_FLIP, lib_path)
from . import stack, float_chain, brute, layout

__all__ = ["conv_acc", "fold", "codes", "maxpool", "join_coeffs", "join_codes",
           "num_threads", "MUTATE_NO_FLIP", "lib_path", "stack", "float_chain",
           "brute", "layout"]
