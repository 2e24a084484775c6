"""CPU oracle of the snapshot-free delta-extraction path.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import, call or load anything in this
package; the product path (paper_2608_00455_amd) never does, and the two
share no code.  Inputs come from the seeded generator in `synth`.

Modules, each following the paper's passage named in its header:
  core   -- step scalars, forward AdamW step, AdamW inversion (sec. 4.1,
            appendix A), BF16 quantisation and detection (sec. 4.2.1); the
            binary32 arithmetic is plain C in dte_oracle.c
  plan   -- transfer plan T (sec. 4.2.2) for the receiver layouts
  remap  -- unravel / containment / ravel (sec. 4.2.2) and direct sparse
            apply (sec. 4.3, eq. direct_sparse_apply)
  run    -- whole-workload driver (seeded state, forward step, detection;
            per-group step scalars, sec. 4.1)
  mcore  -- Megatron-Core sender layout and converter (appendix B,
            eq. mcore_fused_qkv, eq. mcore_tp_shard, eq. qkv_converter):
            detection in the paper's order for one trainer TP rank
  timing, recipe_compare, mode_b -- reports built on the above: the CPU
            baseline's timing, the input recipe's effect, and the
            reconstruction counts when torch.optim.AdamW takes the step

Pins (tests/test_oracle_*.py) tie every function to the paper and to
mathematics outside this package.  Parity unpinned: the change fraction and
reconstruction-mismatch counts of the paper's own training states (not
available), and the choice of binary32 operation order among algebraically
equal forms of the inverse (fixed by reading, see core/dte_oracle.c).
"""
