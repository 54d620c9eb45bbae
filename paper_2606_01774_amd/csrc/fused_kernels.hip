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
    run_chain<Fused<Out, DK, LP>>(a, smem);
}

// The same without the clean outputs: a further noisy view of the complementary-view forward.
template <typename Out, int DK, int LP>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_noisy_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, DK, LP, false, false, float, false, true>>(a, smem);
}

// Noisy blocks of two 32-position sub-blocks (blocks of 34 to 64 positions, even), with and
// without the clean outputs.
template <typename Out, int DK>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_pair_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, DK, 32, false, false, float, false, false, true>>(a, smem);
}
template <typename Out, int DK>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_pair_noisy_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, DK, 32, false, false, float, false, true, true>>(a, smem);
}

// Noisy blocks of 1 .. 8 positions inside 32-position clean chunks.
template <typename Out, int DK>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_small_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, DK, 32, false, false, float, false, false, false, true>>(a, smem);
}

template <typename K>
static hipError_t launch_kernel(void (*kern)(ScanArgs), const ScanArgs &a, hipStream_t s)
{
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  K::BYTES);
    });
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(chain_grid(a)), dim3(K::kThreads), K::BYTES, s, a);
    return hipGetLastError();
}

template <typename Out, int DK, int LP, bool NO_O = false>
static hipError_t launch_one(const ScanArgs &a, hipStream_t s)
{
    typedef Fused<Out, DK, LP, false, false, float, false, NO_O> K;
    return launch_kernel<K>(NO_O ? bdgdn_fwd_pipelined_noisy_kernel<Out, DK, LP> : bdgdn_fwd_pipelined_kernel<Out, DK, LP>,
                            a, s);
}

template <typename Out, int DK, bool NO_O = false>
static hipError_t launch_pair(const ScanArgs &a, hipStream_t s)
{
    typedef Fused<Out, DK, 32, false, false, float, false, NO_O, true> K;
    return launch_kernel<K>(NO_O ? bdgdn_fwd_pipelined_pair_noisy_kernel<Out, DK> : bdgdn_fwd_pipelined_pair_kernel<Out, DK>,
                            a, s);
}

// The same forward that also writes the seed state of every (block, v-head) to a.bs (the
// complementary-view schedule's first pass); d_k = 128.
template <typename Out, int LP>
__global__ void __launch_bounds__(768) bdgdn_fwd_pipelined_seeds_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, 128, LP, false, true>>(a, smem);
}

template <typename Out, int LP>
static hipError_t launch_seeds(const ScanArgs &a, hipStream_t s)
{
    typedef Fused<Out, 128, LP, false, true> K;
    auto kern = bdgdn_fwd_pipelined_seeds_kernel<Out, LP>;
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, K::BYTES);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(chain_grid(a)), dim3(K::kThreads), K::BYTES, s, a);
    return hipGetLastError();
}

hipError_t launch_fwd_pipelined_seeds(Types ty, int lp, const ScanArgs &a, hipStream_t s)
{
    if (!pipelined_supported(ty, 128, lp) || a.n_vt * 32 != a.dv || !a.bs) return hipErrorInvalidValue;
    if (ty == Types::BF16_IN_F32_OUT) return lp == 16 ? launch_seeds<float, 16>(a, s) : launch_seeds<float, 32>(a, s);
    return lp == 16 ? launch_seeds<__bf16, 16>(a, s) : launch_seeds<__bf16, 32>(a, s);
}

bool pipelined_supported(Types ty, int dk, int lp)
{
    return ty != Types::F32 && (dk == 64 || dk == 128) && (lp == 16 || lp == 32);
}

hipError_t launch_fwd_pipelined(Types ty, int dk, int lp, const ScanArgs &a, hipStream_t s, bool clean_out)
{
    if (!pipelined_supported(ty, dk, lp) || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK, LP) \
    if (dk == DK && lp == LP) return clean_out ? launch_one<OUT, DK, LP>(a, s) : launch_one<OUT, DK, LP, true>(a, s);
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64, 16) BDGDN_CASE(float, 64, 32) BDGDN_CASE(float, 128, 16) BDGDN_CASE(float, 128, 32)
    } else {
        BDGDN_CASE(__bf16, 64, 16) BDGDN_CASE(__bf16, 64, 32) BDGDN_CASE(__bf16, 128, 16) BDGDN_CASE(__bf16, 128, 32)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

bool small_supported(Types ty, int dk, int L)
{
    return ty != Types::F32 && (dk == 64 || dk == 128) && L >= 1 && L <= 8 && (L & (L - 1)) == 0;
}

hipError_t launch_fwd_pipelined_small(Types ty, int dk, const ScanArgs &a, hipStream_t s)
{
    if (!small_supported(ty, dk, a.nl) || a.L != 32 || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK)                                                                      \
    if (dk == DK) {                                                                              \
        typedef Fused<OUT, DK, 32, false, false, float, false, false, false, true> K;            \
        return launch_kernel<K>(bdgdn_fwd_pipelined_small_kernel<OUT, DK>, a, s);                \
    }
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64) BDGDN_CASE(float, 128)
    } else {
        BDGDN_CASE(__bf16, 64) BDGDN_CASE(__bf16, 128)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

bool pair_supported(Types ty, int dk, int L)
{
    return ty != Types::F32 && (dk == 64 || dk == 128) && L > 32 && L <= 64 && L % 2 == 0;
}

hipError_t launch_fwd_pipelined_pair(Types ty, int dk, const ScanArgs &a, hipStream_t s, bool clean_out)
{
    if (!pair_supported(ty, dk, 2 * a.L) || a.n_vt * 32 != a.dv) return hipErrorInvalidValue;
#define BDGDN_CASE(OUT, DK) \
    if (dk == DK) return clean_out ? launch_pair<OUT, DK>(a, s) : launch_pair<OUT, DK, true>(a, s);
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_CASE(float, 64) BDGDN_CASE(float, 128)
    } else {
        BDGDN_CASE(__bf16, 64) BDGDN_CASE(__bf16, 128)
    }
#undef BDGDN_CASE
    return hipErrorInvalidValue;
}

}  // namespace bdgdn
