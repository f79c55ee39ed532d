"""DeLS-Spec block drafting on MI355X (gfx950): HIP kernels behind a C ABI (libdels.so).

The compute entry points live in `binding` (combine_logits, draft_block, accept_len);
they load the HIP library on first use and fail if it is missing.  `workloads` holds
the seeded synthetic input generators.
"""
__all__ = ["binding", "workloads"]
