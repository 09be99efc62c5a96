"""Device-side construction of the full-size workloads for the GPU tests.

The packs are drawn on the GPU from seeded generators and laid out in the
packed varlen format plus a paged cache by ``inputs.DevicePack`` (harness
only: it draws and places numbers and holds none of the attention or
log-prob arithmetic).  Rows the oracle needs are copied back to the host.
"""
from paper_2609_35140_amd.inputs import NAN_BF16, DevicePack, host_bits  # noqa: F401
