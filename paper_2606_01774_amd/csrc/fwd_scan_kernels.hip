// fwd_scan_kernels.hip -- the two-kernel training forward:
//   bdgdn_k1_intra_kernel : one workgroup per (block, v-head): the block-local UT
//                           transform and masked Q K^T (intra.hpp), written as one
//                           record per (block, v-head) to the workspace;
//   bdgdn_k2_scan_kernel  : one workgroup per (sequence or document, v-head, d_v
//                           tile): the sequential clean-state scan with each noisy
//                           block evaluated from the on-chip boundary state (scan.hpp).
#include <mutex>

#include "kernels.hpp"
#include "scan.hpp"

namespace bdgdn {

#ifndef BDGDN_INTRA_NW
#define BDGDN_INTRA_NW 4
#endif
constexpr int kScanBV = 32;
constexpr int kIntraNW = BDGDN_INTRA_NW;

template <typename In, int DK, int LP>
__global__ void __launch_bounds__(64 * kIntraNW) bdgdn_k1_intra_kernel(IntraArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Intra<In, DK, LP, kIntraNW> K1;
    typedef typename K1::Row Row;
    const long id = blockIdx.x;
    const long gb = id / a.h_v;           // global block: sequence b, block j of it
    const int h = (int)(id % a.h_v);
    const int b = (int)(gb / a.nblk), j = (int)(gb % a.nblk);
    const long row0 = (long)b * a.T + (long)j * a.L;
    const int nvalid = a.T - j * a.L < a.L ? a.T - j * a.L : a.L;
    const int hq = h / (a.h_v / a.h_qk);
    const long qk_off = (row0 * a.h_qk + hq) * DK;
    const long g_off = row0 * a.h_v + h;
    const Row *src[4] = {static_cast<const Row *>(a.k) + qk_off, static_cast<const Row *>(a.q) + qk_off,
                         static_cast<const Row *>(a.kn) + qk_off, static_cast<const Row *>(a.qn) + qk_off};
    const float *gsrc[4] = {a.g + g_off, a.beta + g_off, a.gn + g_off, a.betan + g_off};
    K1 k1(smem);
    k1.run(src, (long)a.h_qk * DK, gsrc, a.h_v, nvalid, a.ws + (gb * a.h_v + h) * (long)K1::Rc::BYTES);
}

template <typename In, typename Out, int DK, int BV, int LP>
__global__ void __launch_bounds__(640) bdgdn_k2_scan_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Scan<In, Out, DK, BV, LP> K2;
    static_assert(K2::kThreads == 640, "launch bounds");
    // ids i, i+8, i+16, ... of a group carry the d_v tiles of one chain, so they land
    // on one XCD and share its L2 for the q/k rows and the records.
    const int id = blockIdx.x;
    const int per = 8 * a.n_vt;
    const int chain = (id / per) * 8 + (id % 8);
    const int vt = (id % per) / 8;
    if (chain >= a.n_chains) return;
    int seq = chain / a.h_v;
    const int h = chain % a.h_v;
    if (a.n_order > 0) seq = a.order[seq];
    long base, len, gb0;
    if (a.cu) {
        base = a.cu[seq];
        len = (long)a.cu[seq + 1] - base;
        gb0 = base / a.L;
    } else {
        base = (long)seq * a.T;
        len = a.T;
        gb0 = (long)seq * a.nblk;
    }
    const int hq = h / (a.h_v / a.h_qk);
    const int v0 = vt * BV;
    typename K2::Chain c;
    const long qk_off = (base * a.h_qk + hq) * DK;
    const long v_off = (base * a.h_v + h) * a.dv + v0;
    c.p0.k = static_cast<const In *>(a.k) + qk_off;
    c.p0.q = static_cast<const In *>(a.q) + qk_off;
    c.p0.kn = static_cast<const In *>(a.kn) + qk_off;
    c.p0.qn = static_cast<const In *>(a.qn) + qk_off;
    c.p0.v = static_cast<const In *>(a.v) + v_off;
    c.p0.vn = static_cast<const In *>(a.vn) + v_off;
    c.p0.rec = a.ws + (gb0 * a.h_v + h) * (long)K2::Rc::BYTES;
    c.p0.o = static_cast<Out *>(a.o) + v_off;
    c.p0.on = static_cast<Out *>(a.on) + v_off;
    c.qks = a.h_qk * DK;
    c.vst = a.h_v * a.dv;
    c.qk_blk = (long)a.L * c.qks;
    c.v_blk = (long)a.L * c.vst;
    c.rec_blk = (long)a.h_v * K2::Rc::BYTES;
    c.len = len;
    c.L = a.L;
    const long state_off = ((long)seq * a.h_v + h) * DK * a.dv + v0;
    c.h0 = a.h0 ? a.h0 + state_off : nullptr;
    c.ht = a.ht ? a.ht + state_off : nullptr;
    c.dv = a.dv;
    c.scale = a.scale;
    K2 k2(smem);
    k2.run(c);
}

template <typename K>
static hipError_t set_lds_once(K kern, int bytes, std::once_flag &once, hipError_t &err)
{
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    });
    return err;
}

template <typename In, typename Out, int DK, int LP>
static hipError_t launch_pair(const IntraArgs &ia, const ScanArgs &sa, hipStream_t s)
{
    typedef Intra<In, DK, LP, kIntraNW> K1;
    typedef Scan<In, Out, DK, kScanBV, LP> K2;
    static_assert(K1::BYTES <= 160 * 1024 && K2::BYTES <= 160 * 1024, "LDS budget");
    auto k1 = bdgdn_k1_intra_kernel<In, DK, LP>;
    auto k2 = bdgdn_k2_scan_kernel<In, Out, DK, kScanBV, LP>;
    static std::once_flag o1, o2;
    static hipError_t e1 = hipSuccess, e2 = hipSuccess;
    if (set_lds_once(k1, K1::BYTES, o1, e1) != hipSuccess) return e1;
    if (set_lds_once(k2, K2::BYTES, o2, e2) != hipSuccess) return e2;
    hipLaunchKernelGGL(k1, dim3((unsigned)(ia.total_blocks * ia.h_v)), dim3(64 * kIntraNW), K1::BYTES, s, ia);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int grid = (sa.n_chains + 7) / 8 * 8 * sa.n_vt;
    hipLaunchKernelGGL(k2, dim3(grid), dim3(K2::kThreads), K2::BYTES, s, sa);
    return hipGetLastError();
}

template <typename In, int LP> static constexpr size_t rec_bytes()
{
    return Rec<typename Prec<In>::Mid, LP>::BYTES;
}

size_t scan_record_bytes(Types ty, int lp)
{
    const bool f32 = ty == Types::F32;
    if (lp == 16) return f32 ? rec_bytes<float, 16>() : rec_bytes<__bf16, 16>();
    if (lp == 32) return f32 ? rec_bytes<float, 32>() : rec_bytes<__bf16, 32>();
    return f32 ? rec_bytes<float, 64>() : rec_bytes<__bf16, 64>();
}

int scan_tile_v() { return kScanBV; }

hipError_t launch_fwd_scan(Types ty, int dk, int lp, const IntraArgs &ia, const ScanArgs &sa, hipStream_t s)
{
    if (sa.dv % kScanBV || sa.n_vt * kScanBV != sa.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(IN, OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_pair<IN, OUT, DK, LP>(ia, sa, s);
#define BDGDN_LPS(IN, OUT, DK) BDGDN_CASE(IN, OUT, DK, 16) BDGDN_CASE(IN, OUT, DK, 32) BDGDN_CASE(IN, OUT, DK, 64)
    switch (ty) {
    case Types::BF16_IN_F32_OUT:
        BDGDN_LPS(__bf16, float, 64)
        BDGDN_LPS(__bf16, float, 128)
        break;
    case Types::BF16_IN_BF16_OUT:
        BDGDN_LPS(__bf16, __bf16, 64)
        BDGDN_LPS(__bf16, __bf16, 128)
        break;
    case Types::F32:
        BDGDN_CASE(float, float, 64, 16) BDGDN_CASE(float, float, 64, 32)
        BDGDN_CASE(float, float, 128, 16) BDGDN_CASE(float, float, 128, 32)
        break;
    }
#undef BDGDN_LPS
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
