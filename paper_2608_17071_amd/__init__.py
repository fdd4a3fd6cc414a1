"""MI355X (gfx950) BF16 linear layer with a fused residual add, Y = X.W^T + R.

The compute path is the HIP library built from ``csrc/`` (see ``kernelarc``
for the Python binding); ``workloads`` draws the seeded synthetic inputs.
"""
