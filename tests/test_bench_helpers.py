"""Host-side helpers of bench.py: the kernel kind of a profiler kernel name, and
the algorithmic work per kind that the roofline entry divides by kernel time.

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


def test_algorithmic_work_of_the_deep_update():
    # 512-2048-2048-2048-64 at batch 8192: the change products' flops are 2 B n_l n_(l+1)
    # summed over the four layers (the roofline's work per launch is their mean), the
    # forward and hidden-delta products likewise, and all kinds together give the
    # step's 2 B (2 sum n_l n_(l+1) + sum_(l>=1) n_l n_(l+1)) flops (no hidden delta of
    # the inputs).
    sizes, B = (512, 2048, 2048, 2048, 64), 8192
    w = bench.kind_work(sizes, B, False, 7, bench.change_splits)
    pairs = [sizes[l] * sizes[l + 1] for l in range(4)]
    assert w["splitk"][0] == 2 * B * sum(pairs)
    assert w["splitk"][0] / 4 == 39191576576.0
    assert w["forward"][0] + w["output"][0] == 2 * B * sum(pairs)
    assert w["backward"][0] == 2 * B * sum(pairs[1:])
    gemm = w["forward"][0] + w["output"][0] + w["backward"][0] + w["splitk"][0]
    assert gemm == 2 * B * (2 * sum(pairs) + sum(pairs[1:]))
    # the change kind's bytes: both operands read once, W and V read and written
    assert w["splitk"][1] == sum(4 * (B * sizes[l] + B * sizes[l + 1]) + 16 * pairs[l] for l in range(4))


def test_algorithmic_bytes_of_the_fused_small_update():
    # 203-120-26, 7 active inputs, batch 512: 16 B per weight (W and V read and written)
    # plus 4 (7 + 26) B per pattern (indices and targets) = 442,016 + 67,584 = 509,600 B.
    w = bench.kind_work((203, 120, 26), 512, True, 7, bench.change_splits)
    assert set(w) == {"fused_fb", "fused_update"}
    assert w["fused_update"][1] == 16 * (204 * 120 + 121 * 26) == 442016
    assert w["fused_fb"][1] == 4 * 512 * (7 + 26) == 67584
    assert w["fused_update"][1] + w["fused_fb"][1] == 509600
