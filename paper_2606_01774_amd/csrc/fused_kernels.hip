// fused_kernels.hip -- the one-kernel training forward (fused.hpp): one workgroup per
// (sequence or document, v-head, 32-column d_v tile) computes each block's UT transform
// and scans the blocks with the noisy stream evaluated from the on-chip boundary state.
#include <mutex>

#include "fused.hpp"
#include "kernels.hpp"

namespace bdgdn {

template <typename Out, int DK, int LP>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Fused<Out, DK, LP> K;
    static_assert(K::kThreads == 768, "launch bounds");
    typedef typename K::In In;
    // ids i, i+8, i+16, ... of a group carry the d_v tiles of one chain, so they land
    // on one XCD and share its L2 for the q/k rows and gates.
    const int id = blockIdx.x;
    const int per = 8 * a.n_vt;
    const int chain = (id / per) * 8 + (id % 8);
    const int vt = (id % per) / 8;
    if (chain >= a.n_chains) return;
    int seq = chain / a.h_v;
    const int h = chain % a.h_v;
    if (a.n_order > 0) seq = a.order[seq];
    long base, len;
    if (a.cu) {
        base = a.cu[seq];
        len = (long)a.cu[seq + 1] - base;
    } else {
        base = (long)seq * a.T;
        len = a.T;
    }
    const int hq = h / (a.h_v / a.h_qk);
    const int v0 = vt * K::BV;
    typename K::Chain c;
    const long qk_off = (base * a.h_qk + hq) * DK;
    const long v_off = (base * a.h_v + h) * a.dv + v0;
    const long g_off = base * a.h_v + h;
    c.p0.k = static_cast<const In *>(a.k) + qk_off;
    c.p0.q = static_cast<const In *>(a.q) + qk_off;
    c.p0.kn = static_cast<const In *>(a.kn) + qk_off;
    c.p0.qn = static_cast<const In *>(a.qn) + qk_off;
    c.p0.v = static_cast<const In *>(a.v) + v_off;
    c.p0.vn = static_cast<const In *>(a.vn) + v_off;
    c.p0.g = a.g + g_off;
    c.p0.beta = a.beta + g_off;
    c.p0.gn = a.gn + g_off;
    c.p0.betan = a.betan + g_off;
    c.p0.o = static_cast<Out *>(a.o) + v_off;
    c.p0.on = static_cast<Out *>(a.on) + v_off;
    c.qks = a.h_qk * DK;
    c.vst = a.h_v * a.dv;
    c.gst = a.h_v;
    c.qk_blk = (long)a.L * c.qks;
    c.v_blk = (long)a.L * c.vst;
    c.g_blk = (long)a.L * c.gst;
    c.len = len;
    c.L = a.L;
    const long state_off = ((long)seq * a.h_v + h) * DK * a.dv + v0;
    c.h0 = a.h0 ? a.h0 + state_off : nullptr;
    c.ht = a.ht ? a.ht + state_off : nullptr;
    c.dv = a.dv;
    c.scale = a.scale;
    K k(smem);
    k.run(c);
}

template <typename Out, int DK, int LP>
static hipError_t launch_one(const ScanArgs &a, hipStream_t s)
{
    typedef Fused<Out, DK, LP> K;
    auto kern = bdgdn_fwd_pipelined_kernel<Out, DK, LP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  K::BYTES);
    });
    if (err != hipSuccess) return err;
    const int grid = (a.n_chains + 7) / 8 * 8 * a.n_vt;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(K::kThreads), K::BYTES, s, a);
    return hipGetLastError();
}

bool pipelined_supported(Types ty, int dk, int lp)
{
    return ty != Types::F32 && (dk == 64 || dk == 128) && (lp == 16 || lp == 32);
}

hipError_t launch_fwd_pipelined(Types ty, int dk, int lp, const ScanArgs &a, hipStream_t s)
{
    if (!pipelined_supported(ty, dk, lp) || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_one<OUT, DK, LP>(a, s);
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64, 16) BDGDN_CASE(float, 64, 32) BDGDN_CASE(float, 128, 16) BDGDN_CASE(float, 128, 32)
    } else {
        BDGDN_CASE(__bf16, 64, 16) BDGDN_CASE(__bf16, 64, 32) BDGDN_CASE(__bf16, 128, 16) BDGDN_CASE(__bf16, 128, 32)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
