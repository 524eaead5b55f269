"""CPU oracle for the one-GPU share of a Dynamic Sequence Parallelism block.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only the test suite, the smoke check and the CPU-baseline leg of
the benchmark use it.  It shares no code with the HIP library and imports
nothing from it.

Everything here is plain, slow and written from the paper's definitions in
float64 NumPy (library matmul and erf as the only primitives):

* ``switch`` / ``unswitch`` / ``exchange_unpack`` -- the Switch primitive of
  the primitive table in the Dynamic Primitives section (Eq. 10) restricted to
  one GPU's share: a layout permute plus a pack into per-destination chunks,
  done on raw bit patterns, for K = 2 or 3 sequence dimensions.
* ``split`` / ``gather`` -- the table's Split and Gather rows (one rank's
  slice; the concatenation of every rank's slice).
* ``attention`` -- scaled dot-product attention, Eq. (3), applied per head
  (Eq. 1-2) along one sequence dimension of a multi-dimensional sequence
  (Eq. 7-8): ``spatial_attention`` over S within each frame and
  ``temporal_attention`` over T at each location.
* ``attention_grouped`` / ``attention_grouped_bwd`` -- grouped key/value
  heads (multi-query, grouped-query) and separate query and key lengths
  (cross-attention), the variants the paper states compatibility with.
* ``attention_bwd`` / ``attention_lse`` -- the backward of attention (the
  chain rule through the softmax) and the row logsumexp it uses.
* ``layernorm``, ``linear``, ``gelu`` and the composites ``st_block`` (the
  full spatial-temporal block) and ``tiny_chain``.
* ``linear_bwd``, ``layernorm_bwd``, ``gelu_bwd``, ``relu_bwd`` and
  ``st_block_bwd`` -- the chain rule through the block, in reverse order.

Pins: every function is checked in ``tests/test_oracle_pins.py`` against
closed forms, invariants, hand-worked fixtures and brute force; see the header
of each module for what pins it.
"""
from .switch import switch, unswitch, exchange_unpack, switch_index_map, split, gather
from .attention import attention, attention_rows, spatial_attention, temporal_attention, \
    temporal_attention_strided, attention_grouped
from .backward import attention_bwd, attention_bwd_units, attention_lse, attention_lse_units, \
    attention_delta_units, attention_grouped_bwd
from .block_bwd import linear_bwd, layernorm_bwd, gelu_bwd, relu_bwd, st_block_bwd
from .block import layernorm, linear, gelu, relu, st_block, tiny_chain, BLOCK_NO_MLP_LN, BLOCK_POST_LN, \
    BLOCK_RELU

__all__ = ["switch", "unswitch", "exchange_unpack", "switch_index_map", "split", "gather", "attention",
           "attention_rows", "spatial_attention", "temporal_attention",
           "temporal_attention_strided", "layernorm", "linear", "gelu", "st_block", "tiny_chain",
           "BLOCK_NO_MLP_LN", "BLOCK_POST_LN", "BLOCK_RELU", "relu", "attention_bwd",
           "attention_bwd_units", "attention_lse", "attention_lse_units", "attention_delta_units",
           "linear_bwd", "layernorm_bwd", "gelu_bwd", "relu_bwd", "st_block_bwd", "attention_grouped",
           "attention_grouped_bwd"]
