"""EntropyInfer prefill hot path on MI355X (gfx950): entropy probe, head
classification and budgeted top-k block selection, block-sparse causal GQA
attention, and a dense causal baseline, behind the C ABI of libentropyinfer.so.

The HIP library is loaded on first use by :mod:`paper_2606_09508_amd.binding`;
importing the package does not touch the GPU.
"""
