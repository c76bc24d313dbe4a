"""Host-side helpers of bench.py: the kernel kind of a profiler kernel name.

rocprofv3 names a template instance with every template argument, defaults
included (the thread count after the epilogue of gemm_kernel), so the kind is
read from the epilogue argument wherever it stands.  A kind that is not
recognised drops that kernel's HBM traffic from the counter summaries.
"""
import bench

NS = "bpk::(anonymous namespace)::"


def test_kernel_kinds_from_profiler_names():
    cases = {
        f"void {NS}gemm_kernel<256, 256, 32, false, false, true, true, {NS}EpiSigmoid, 512>"
        f"(float const*, int, float const*, int, int, int, int, int, {NS}EpiSigmoid)": "forward",
        f"void {NS}gemm_kernel<128, 64, 32, false, false, true, true, {NS}EpiPartial, 256>(float const*)": "output",
        f"void {NS}gemm_kernel<64, 64, 32, false, false, true, false, {NS}EpiOutputDelta, 256>(float const*)":
            "output",
        f"void {NS}gemm_kernel<256, 256, 32, false, true, true, true, {NS}EpiHiddenDelta, 512>(float const*)":
            "backward",
        f"void {NS}gemm_kernel<128, 128, 32, true, false, true, true, {NS}EpiUpdate, 256>(float const*)": "change",
        f"void {NS}gemm_kernel<128, 128, 32, true, false, true, true, {NS}EpiSplitUpdate, 256>(float const*)":
            "splitk",
        f"void {NS}skinny_kernel<2, true, false, false, false, false, {NS}EpiSplitUpdate>"
        f"(float const*, int, float const*, int, int, int, int, int, {NS}EpiSplitUpdate, {NS}CtxInput)": "splitk",
        f"void {NS}skinny_kernel<1, false, false, true, true, false, {NS}EpiSigmoid>(float const*)": "forward",
        f"{NS}bias_update_kernel(bpk::BiasJobs, float, float, float, unsigned long long*)": "bias",
        f"{NS}output_finish_kernel(float const*, int, unsigned long, int, int, int)": "output_finish",
        f"void {NS}elman_window_kernel<1, 4, 1>(bpk::ElmanWindow)": "seq_win",
        f"void {NS}small_update_kernel<false, 512>(int const*, int)": "fused_update",
        f"void {NS}small_fwdbwd_kernel<2, false, 128, 32>(int const*, int)": "fused_fb",
        f"{NS}sse_reduce_kernel(double const*, int, double*)": "reduce",
        "__amd_rocclr_fillBufferAligned": None,
    }
    for name, kind in cases.items():
        assert bench.kind_of_kernel(name) == kind, name
