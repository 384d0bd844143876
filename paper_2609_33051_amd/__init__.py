"""SketchSSM decode hot path for MI355X (gfx950).

Submodules:
  binding  -- ctypes binding of the C-ABI library libsketchssm.so
              (sketchssm_update / sketchssm_decode / sketchssm_full_read_baseline)
  layer    -- device buffers of one linear-attention layer and its decode loop
  inputs   -- seeded synthetic workloads
  traffic  -- byte accounting (the paper's model and this implementation's)

Nothing is imported eagerly: importing the package does not load the HIP library.
"""
