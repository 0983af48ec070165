"""fp64 CPU oracle of the SMem attention path -- test infrastructure only.

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the product path."""
from .smem_oracle import *  # noqa: F401,F403
from .smem_oracle import (Store, StoreError, encode_blocks, encode_into_store,  # noqa: F401
                          reader_prefill_block, reader_decode, softmax_read, rel_err,
                          MASK_BIDIR, MASK_CAUSAL, EEXIST, ENOENT, EINVAL)
