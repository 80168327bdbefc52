"""eDKM hot path on MI355X: uniquified DKM weight clustering, forward and backward.

Submodules:
  edkm     — ctypes binding of the C-ABI library ``libedkm.so`` (HIP, gfx950).
  function — ``dkm(w, c0, ...)``: the clustering as a differentiable torch op.
  runner   — one init_unique + forward (+ backward) call with outputs allocated.
  inputs   — seeded synthetic inputs (weights, initial centroids, gradients).

Importing the package does not load the HIP library; ``edkm`` does, and fails
loudly if it is missing.
"""
