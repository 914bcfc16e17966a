"""delta-Vision visual-memory path for MI355X (gfx950).

Per-layer low-rank adapters build each layer's visual memory from the shared
visual embeddings (Section 3.1, Eq. 4-5), the memory is normalised and
projected by the frozen per-layer K/V weights (Section 3.2, Eq. 7), and text
queries attend over all visual keys plus their own causal context (Section 3.2,
Eq. 9). The arithmetic runs in hand-written HIP kernels behind the C ABI of
``include/deltavision.h``; this package only marshals tensors into it.
"""
from ._lib import (ACT_GELU, ACT_SILU, ATTENTION_SCRATCH_BYTES, KERNEL_ATTENTION, KERNEL_DELTA_PREP, KERNEL_DELTA_SCAN,
                   KERNEL_DOWN, KERNEL_KV, KERNEL_UP,
                   PROBE_BLOCKS, PROBE_FLOP_PER_ITER,
                   DeltaVisionError, KVEpilogue, build_visual_memory, delta_rule_workspace,
                   delta_rule_write, kept_visual_kv,
                   kept_visual_kv_workspace, load, probe_mfma, project_visual_kv,
                   project_visual_kv_fused, set_fused_kv, set_up_kernel, project_visual_kv_up_kernel,
                   project_visual_kv_ex_workspace,
                   project_visual_kv_workspace, recurrent_visual_kv,
                   recurrent_visual_kv_workspace, text_visual_attention,
                   text_visual_attention_noalloc, text_visual_attention_workspace, time_kernel)

__all__ = [
    "ACT_SILU", "ACT_GELU", "DeltaVisionError", "load", "build_visual_memory",
    "project_visual_kv", "project_visual_kv_workspace", "project_visual_kv_fused", "set_fused_kv", "set_up_kernel", "project_visual_kv_up_kernel", "project_visual_kv_ex_workspace",
    "KVEpilogue", "recurrent_visual_kv",
    "recurrent_visual_kv_workspace", "kept_visual_kv", "kept_visual_kv_workspace",
    "text_visual_attention", "text_visual_attention_noalloc", "ATTENTION_SCRATCH_BYTES",
    "text_visual_attention_workspace", "time_kernel", "KERNEL_DOWN", "KERNEL_UP", "KERNEL_KV",
    "KERNEL_ATTENTION", "KERNEL_DELTA_PREP", "KERNEL_DELTA_SCAN", "delta_rule_write",
    "delta_rule_workspace", "probe_mfma", "PROBE_BLOCKS", "PROBE_FLOP_PER_ITER",
]
