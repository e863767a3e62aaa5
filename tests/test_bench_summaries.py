"""Host-side logic of bench.py's profile summaries (CPU only)."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _rows(names):
    return [{"Dispatch_Id": str(i), "Kernel_Name": n} for i, n in enumerate(names)]


def test_classify_dispatches_plain_layer():
    seq = ["modnorm_kernel", "gemm_bf16_kernel<A,0>", "attention_bf16_kernel", "gemm_bf16_kernel<B,2>",
           "modnorm_kernel", "gemm_bf16_kernel<C,1>", "gemm_bf16_kernel<D,2>",
           "modnorm_kernel", "gemm_bf16_kernel<A,0>"]
    role = bench._classify_dispatches(_rows(seq))
    assert [role[i] for i in range(len(seq))] == ["modnorm", "gemm_qkv", "attention", "gemm_o", "modnorm",
                                                  "gemm_up", "gemm_down", "modnorm", "gemm_qkv"]


def test_classify_dispatches_split_products_with_fused_norms():
    # Small batch: split keys (merge), split output and MLP-down products
    # whose slice reductions also take the following norm (no modnorm launch).
    seq = ["modnorm_kernel", "gemm_bf16_kernel<A,0>", "attention_bf16_kernel", "attn_merge_kernel",
           "gemm_bf16_kernel<B,3>", "gemm_split_reduce_norm_kernel<8>", "gemm_bf16_kernel<C,1>",
           "gemm_bf16_kernel<D,3>", "gemm_split_reduce_norm_kernel<8>", "gemm_bf16_kernel<A,0>",
           "attention_bf16_kernel"]
    role = bench._classify_dispatches(_rows(seq))
    assert [role[i] for i in range(len(seq))] == ["modnorm", "gemm_qkv", "attention", "attn_merge", "gemm_o",
                                                  "gemm_o", "gemm_up", "gemm_down", "gemm_down", "gemm_qkv",
                                                  "attention"]


def test_classify_dispatches_deferred_norms():
    # Large batch: unsplit output and MLP-down products leave the norm to the
    # product after them (no modnorm launch between layers), and the call's
    # shift-table kernel and the final norm sit outside the projections.
    seq = ["shift_proj_kernel", "in_proj_kernel", "modnorm_kernel", "gemm_bf16_kernel<A,0,false>",
           "attention_bf16_kernel", "gemm_bf16_kernel<B,2,true>", "gemm_bf16_kernel<C,1,true>",
           "gemm_bf16_kernel<D,2,true>", "gemm_bf16_kernel<A,0,true>", "attention_bf16_kernel",
           "gemm_bf16_kernel<B,2,true>", "gemm_bf16_kernel<C,1,true>", "gemm_bf16_kernel<D,2,false>",
           "modnorm_kernel", "out_proj_euler_kernel", "in_proj_kernel", "modnorm_kernel",
           "gemm_bf16_kernel<A,0,false>"]
    role = bench._classify_dispatches(_rows(seq))
    assert [role[i] for i in range(len(seq))] == ["other", "other", "modnorm", "gemm_qkv", "attention", "gemm_o",
                                                  "gemm_up", "gemm_down", "gemm_qkv", "attention", "gemm_o",
                                                  "gemm_up", "gemm_down", "modnorm", "other", "other", "modnorm",
                                                  "gemm_qkv"]


def test_visible_keys_counts_the_prefix_lm_mask():
    # brute force over the mask: token t sees key j iff j < max(P - c, t + 1)
    for P in (1, 5, 17):
        for c in range(P + 1):
            brute = sum(1 for t in range(P) for j in range(P) if j < max(P - c, t + 1))
            assert bench.visible_keys(P, c) == brute
