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

template <typename Out, int DK, int LP>
__global__ void __launch_bounds__(64 * (DK / 16 + 2 + kOutStagers)) bdgdn_chunk_out_kernel(ChunkArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_segment<OutKernel<Out, DK, LP, kOutStagers>>(a, smem);
}

size_t chunk_rec_bytes(int lp) { return lp <= 16 ? CRec<16>::BYTES : CRec<32>::BYTES; }

bool chunked_supported(Types ty, int dk, int dv, int lp)
{
    return ty != Types::F32 && dk == dv && (dk == 64 || dk == 128) && (lp == 16 || lp == 32);
}

template <typename Out, int DK, int LP>
static hipError_t launch_chunked(const ChunkArgs &a, hipStream_t s)
{
    typedef OutKernel<Out, DK, LP, kOutStagers> KO;
    typedef StatesKernel<DK, LP> KS;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(bdgdn_chunk_out_kernel<Out, DK, LP>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, KO::BYTES);
        if (err == hipSuccess)
            err = hipFuncSetAttribute(reinterpret_cast<const void *>(bdgdn_chunk_states_kernel<DK, LP>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, KS::BYTES);
    });
    if (err != hipSuccess) return err;
    if (a.n1 > 0 && a.J_max > 0) {
        const long rec_units = (long)a.n1 * a.h_v * a.J_max;
        auto krec = bdgdn_chunk_rec_kernel<DK, LP>;
        constexpr int kRecBytes = RecKernel<DK, LP>::BYTES;
        hipLaunchKernelGGL(krec, dim3((unsigned)((rec_units + 3) / 4)), dim3(256), kRecBytes, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        auto kst = bdgdn_chunk_states_kernel<DK, LP>;
        hipLaunchKernelGGL(kst, dim3((unsigned)(a.n1 * a.h_v * a.n_vt)), dim3(256), KS::BYTES, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.n_units <= 0) return hipSuccess;
    auto kout = bdgdn_chunk_out_kernel<Out, DK, LP>;
    hipLaunchKernelGGL(kout, dim3((unsigned)a.n_units), dim3(KO::kThreads), KO::BYTES, s, a);
    return hipGetLastError();
}

hipError_t launch_fwd_chunked(Types ty, int dk, int lp, const ChunkArgs &a, hipStream_t s)
{
    if (!chunked_supported(ty, dk, a.dv, lp) || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_chunked<OUT, DK, LP>(a, s);
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64, 16) BDGDN_CASE(float, 64, 32) BDGDN_CASE(float, 128, 16) BDGDN_CASE(float, 128, 32)
    } else {
        BDGDN_CASE(__bf16, 64, 16) BDGDN_CASE(__bf16, 64, 32) BDGDN_CASE(__bf16, 128, 16) BDGDN_CASE(__bf16, 128, 32)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
