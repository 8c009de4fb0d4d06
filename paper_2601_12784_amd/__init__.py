"""MI355X-native paged decode attention for skewed rollout batches.

The compute path is a C-ABI HIP library (libsf_decode_attn.so, built for
gfx950); paper_2601_12784_amd.binding marshals torch tensors into it.
paper_2601_12784_amd.workloads draws the seeded synthetic batches.
"""
