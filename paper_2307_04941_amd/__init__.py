"""MI355X (gfx950) forward 2-D convolution as an implicit matrix product on
fp32 MFMA, after MG3MConv (arXiv 2307.04941).

The compute path is libmg3m.so (HIP kernels + C ABI, see include/mg3m.h);
``paper_2307_04941_amd.mg3m`` is its thin Python binding.  Names are loaded
lazily so that importing the package does not load the HIP library.
"""

_EXPORTS = {
    "conv2d_fwd", "conv2d_fwd_f32", "conv2d_fwd_f32_ex", "conv2d_out_dims",
    "conv2d_out_dims_hw", "conv2d_fwd_f32_hw", "conv2d_fwd_f32_hw_workspace_bytes",
    "conv2d_fwd_f32_acc64", "conv2d_fwd_f32_acc64_plan_string", "conv2d_fwd_f32_fused",
    "maxpool2d_f32", "maxpool2d_out_dims", "maxpool2d", "Net", "Layer",
    "conv2d_fwd_f32_workspace_bytes", "conv2d_fwd_f32_plan_string",
    "conv2d_fwd_f32_plan_info", "mg3m_padding_overhead", "mg3m_time_next_kernel", "mg3m_status_string",
    "mg3m_last_error", "load_library", "Mg3mError", "HWCN", "NCHW",
}


def __getattr__(name):
    if name in _EXPORTS:
        from . import mg3m
        return getattr(mg3m, name)
    raise AttributeError(name)
