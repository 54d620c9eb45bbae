// chunked_kernels.hip -- launchers of the chunk-parallel training forward (chunked.hpp):
// the clean UT records and the state pass over the blocks before each chain's last
// segment (skipped when every chain is one segment), then one workgroup per (chain,
// segment) for the outputs.
#include <mutex>

#include "chunked.hpp"
#include "kernels.hpp"

namespace bdgdn {

using namespace chunked;

constexpr int kOutStagers = 4;

template <int DK, int LP>
__global__ void __launch_bounds__(256) bdgdn_chunk_rec_kernel(ChunkArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    RecKernel<DK, LP>::run(a, smem);
}

template <int DK, int LP>
__global__ void __launch_bounds__(256) bdgdn_chunk_states_kernel(ChunkArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    StatesKernel<DK, LP>::run(a, smem);
}

template <typename Out, int DK, int DV, int LP>
__global__ void __launch_bounds__(64 * (DV / 16 + 2 + kOutStagers)) bdgdn_chunk_out_kernel(ChunkArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_segment<OutKernel<Out, DK, DV, LP, kOutStagers>>(a, smem);
}

bool chunk_tile_supported(int dk, int tile) { return tile == dk || tile == 32; }

size_t chunk_rec_bytes(int lp) { return lp <= 16 ? CRec<16>::BYTES : CRec<32>::BYTES; }

bool chunked_supported(Types ty, int dk, int dv, int lp)
{
    return ty != Types::F32 && dk == dv && (dk == 64 || dk == 128) && (lp == 16 || lp == 32);
}

template <typename Out, int DK, int DV, int LP>
static hipError_t launch_chunked(const ChunkArgs &a, hipStream_t s)
{
    typedef OutKernel<Out, DK, DV, LP, kOutStagers> KO;
    typedef StatesKernel<DK, LP> KS;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(bdgdn_chunk_out_kernel<Out, DK, DV, LP>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, KO::BYTES);
        if (err == hipSuccess)
            err = hipFuncSetAttribute(reinterpret_cast<const void *>(bdgdn_chunk_states_kernel<DK, LP>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, KS::BYTES);
        if (err == hipSuccess)
            err = hipFuncSetAttribute(reinterpret_cast<const void *>(bdgdn_chunk_rec_kernel<DK, LP>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, RecKernel<DK, LP>::BYTES);
    });
    if (err != hipSuccess) return err;
    if (a.n1 > 0 && a.J_max > 0) {
        typedef RecKernel<DK, LP> KR;
        const int np = (a.n1 * a.h_v + 7) & ~7;   // chains padded to the eight XCDs
        const long rec_groups = (long)np * ((a.J_max + KR::kWaves - 1) / KR::kWaves);
        auto krec = bdgdn_chunk_rec_kernel<DK, LP>;
        constexpr int kRecBytes = KR::BYTES;
        hipLaunchKernelGGL(krec, dim3((unsigned)rec_groups), dim3(KR::kThreads), kRecBytes, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        auto kst = bdgdn_chunk_states_kernel<DK, LP>;
        hipLaunchKernelGGL(kst, dim3((unsigned)(np * a.n_vt)), dim3(256), KS::BYTES, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.n_groups <= 0) return hipSuccess;
    const long n_wg = (long)(a.n_groups + 7) / 8 * 8 * (a.h_v / a.h_qk) * a.n_ot;
    auto kout = bdgdn_chunk_out_kernel<Out, DK, DV, LP>;
    hipLaunchKernelGGL(kout, dim3((unsigned)n_wg), dim3(KO::kThreads), KO::BYTES, s, a);
    return hipGetLastError();
}

hipError_t launch_fwd_chunked(Types ty, int dk, int lp, const ChunkArgs &a, hipStream_t s)
{
    if (!chunked_supported(ty, dk, a.dv, lp) || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
    const int tile = a.dv / a.n_ot;
    if (!chunk_tile_supported(dk, tile) || tile * a.n_ot != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK, LP) \
    if (dk == DK && lp == LP)                                                             \
        return tile == DK ? launch_chunked<OUT, DK, DK, LP>(a, s) : launch_chunked<OUT, DK, 32, LP>(a, s);
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64, 16) BDGDN_CASE(float, 64, 32) BDGDN_CASE(float, 128, 16) BDGDN_CASE(float, 128, 32)
    } else {
        BDGDN_CASE(__bf16, 64, 16) BDGDN_CASE(__bf16, 64, 32) BDGDN_CASE(__bf16, 128, 16) BDGDN_CASE(__bf16, 128, 32)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
