// fwd_kernels.hip -- the fused two-stream training forward (one workgroup per
// (sequence or document, v-head, d_v tile)).  The clean state stays in registers
// across the sequential block loop; each noisy block is evaluated from the
// in-register boundary state and never materialised (Appendix "Route II: Fused
// Two-Stream", Algorithm route-twostream-fwd), here with the clean state advanced by
// whole blocks through the block-local UT transform (eq. f-blk).
#include <mutex>

#include "engine.hpp"
#include "kernels.hpp"

namespace bdgdn {

#ifndef BDGDN_FWD_BV
#define BDGDN_FWD_BV 32
#endif
#ifndef BDGDN_FWD_NW
#define BDGDN_FWD_NW 8
#endif
constexpr int kFwdBV = BDGDN_FWD_BV;  // d_v columns per workgroup
constexpr int kFwdNW = BDGDN_FWD_NW;  // waves per workgroup
constexpr int kFwdThreads = 64 * kFwdNW;

template <typename In, typename Op, typename Out, int DK, int BV, int LP>
__global__ void __launch_bounds__(kFwdThreads) bdgdn_fwd_fused_kernel(FwdArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Engine<In, Op, Out, DK, BV, LP, true, true, true, kFwdNW> Eng;
    // Workgroup ids are dealt round-robin over the 8 XCDs; ids i, i+8, i+16, ... of a
    // group carry the d_v tiles of one chain so they share that XCD's L2 for q/k.
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
    const int v0 = vt * BV;
    Eng eng(smem);
    f32x4 S[Eng::NSW];
    const long state_off = ((long)seq * a.h_v + h) * DK * a.dv + v0;
    eng.load_state(S, a.h0 ? a.h0 + state_off : nullptr, a.dv);
    eng.write_st(S);
    __syncthreads();
    // Block descriptors are rebuilt by value each iteration (scalar arithmetic); an
    // array of them indexed at run time would live in scratch memory.
    auto make_io = [&](long j0) {
        typename Eng::IO x;
        const long row0 = base + j0;
        const long qk_off = (row0 * a.h_qk + hq) * DK;
        const long v_off = (row0 * a.h_v + h) * a.dv + v0;
        const long g_off = row0 * a.h_v + h;
        x.qk_stride = (long)a.h_qk * DK;
        x.v_stride = (long)a.h_v * a.dv;
        x.gate_stride = a.h_v;
        x.k = static_cast<const In *>(a.k) + qk_off;
        x.q = static_cast<const In *>(a.q) + qk_off;
        x.v = static_cast<const In *>(a.v) + v_off;
        x.kn = static_cast<const In *>(a.kn) + qk_off;
        x.qn = static_cast<const In *>(a.qn) + qk_off;
        x.vn = static_cast<const In *>(a.vn) + v_off;
        x.g = a.g + g_off;
        x.beta = a.beta + g_off;
        x.gn = a.gn + g_off;
        x.betan = a.betan + g_off;
        x.o = static_cast<Out *>(a.o) + v_off;
        x.on = static_cast<Out *>(a.on) + v_off;
        x.nvalid = (int)(len - j0 < a.L ? len - j0 : a.L);
        return x;
    };
    typename Eng::Fetched f;
    if (len > 0) eng.fetch(make_io(0), f);
    for (long j0 = 0; j0 < len; j0 += a.L) {
        const bool more = j0 + a.L < len;
        eng.step(make_io(j0), more, make_io(more ? j0 + a.L : j0), f, S, a.scale);
    }
    if (a.ht) eng.store_state(S, a.ht + state_off, a.dv);
}

template <typename In, typename Op, typename Out, int DK, int LP>
static hipError_t launch_one(const FwdArgs &a, hipStream_t s)
{
    typedef Layout<Op, DK, kFwdBV, LP, true, true, true> Ly;
    static_assert(Ly::BYTES <= 160 * 1024, "LDS budget");
    auto kern = bdgdn_fwd_fused_kernel<In, Op, Out, DK, kFwdBV, LP>;
    static std::once_flag once;
    static hipError_t attr_err = hipSuccess;
    std::call_once(once, [&] {
        attr_err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, Ly::BYTES);
    });
    if (attr_err != hipSuccess) return attr_err;
    const int groups = (a.n_chains + 7) / 8;
    const int grid = groups * 8 * a.n_vt;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kFwdThreads), Ly::BYTES, s, a);
    return hipGetLastError();
}

int fwd_tile_v() { return kFwdBV; }

bool fwd_supported(Types ty, int dk, int lp)
{
    (void)dk;
    return ty != Types::F32 || lp <= 32;
}

hipError_t launch_fwd_fused(Types ty, int dk, int lp, const FwdArgs &a, hipStream_t s)
{
    if (a.dv % kFwdBV || a.n_vt * kFwdBV != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(IN, OP, OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_one<IN, OP, OUT, DK, LP>(a, s);
#define BDGDN_LPS(IN, OP, OUT, DK) \
    BDGDN_CASE(IN, OP, OUT, DK, 16) BDGDN_CASE(IN, OP, OUT, DK, 32) BDGDN_CASE(IN, OP, OUT, DK, 64)
    switch (ty) {
    case Types::BF16_IN_F32_OUT:
        BDGDN_LPS(__bf16, _Float16, float, 64)
        BDGDN_LPS(__bf16, _Float16, float, 128)
        break;
    case Types::BF16_IN_BF16_OUT:
        BDGDN_LPS(__bf16, _Float16, __bf16, 64)
        BDGDN_LPS(__bf16, _Float16, __bf16, 128)
        break;
    case Types::F32:
        BDGDN_CASE(float, float, float, 64, 16) BDGDN_CASE(float, float, float, 64, 32)
        BDGDN_CASE(float, float, float, 128, 16) BDGDN_CASE(float, float, float, 128, 32)
        break;
    }
#undef BDGDN_LPS
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
