// split_kernels.hip -- the split schedule of the two-stream training forward (Appendix
// "Route I": the clean scan hands each noisy block its seed state through HBM, and a
// separate kernel evaluates the noisy blocks, all in parallel):
//   K2  bdgdn_k2_scan_states_kernel  the one-kernel clean scan (fused.hpp, SPLIT) writing
//                                    the clean state before every block, fp32, indexed by
//                                    (global block, v-head), plus the clean outputs;
//   K3  bdgdn_k3_noisy_kernel        the block-end readout of every noisy block from its
//                                    seed state (serve.hpp, the same pass as denoise).
// It exists to attribute the noisy pass to a kernel of its own and as an equivalence check
// of the fused schedule; the workspace holds one 64 KiB state per (block, v-head).
#include <mutex>

#include "fused.hpp"
#include "kernels.hpp"
#include "serve.hpp"

namespace bdgdn {

template <typename Out, int LP, typename SeedT = float, bool STATES = false>
__global__ void __launch_bounds__(768) bdgdn_k2_scan_states_kernel(ScanArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    run_chain<Fused<Out, 128, LP, true, true, SeedT, STATES>>(a, smem);
}

template <typename Out, int LP>
__global__ void __launch_bounds__(256) bdgdn_k3_noisy_kernel(NoisyArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Serve<Out, 128, LP, false, false> K;
    typedef typename K::In In;
    const long gblk = blockIdx.x / a.h_v;
    const int h = blockIdx.x % a.h_v;
    long row0;
    int nvalid;
    if (a.cu) {
        // the document holding the block: the last d < N with cu[d] <= row0 (documents
        // start on block boundaries, so it contains the whole block)
        row0 = gblk * a.L;
        int lo = 0, hi = a.n_docs;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.cu[mid] <= row0)
                lo = mid;
            else
                hi = mid;
        }
        const long rem = (long)a.cu[lo + 1] - row0;
        nvalid = rem < a.L ? (int)rem : a.L;
    } else {
        const long b = gblk / a.nblk;
        const int j = (int)(gblk % a.nblk);
        row0 = b * a.T + (long)j * a.L;
        const int rem = a.T - j * a.L;
        nvalid = rem < a.L ? rem : a.L;
    }
    const int hq = h / (a.h_v / a.h_qk);
    typename K::Unit u;
    const long qk_off = (row0 * a.h_qk + hq) * 128;
    const long v_off = (row0 * a.h_v + h) * 128;
    u.k = static_cast<const In *>(a.kn) + qk_off;
    u.q = static_cast<const In *>(a.qn) + qk_off;
    u.v = static_cast<const In *>(a.vn) + v_off;
    u.g = a.gn + row0 * a.h_v + h;
    u.beta = a.betan + row0 * a.h_v + h;
    u.state = const_cast<float *>(a.bs) + (gblk * a.h_v + h) * 128 * 128;   // only read
    u.o = static_cast<Out *>(a.on) + v_off;
    u.qks = a.h_qk * 128;
    u.vst = a.h_v * 128;
    u.gst = a.h_v;
    u.nvalid = nvalid;
    u.scale = a.scale;
    K k(smem);
    k.run(u);
}

template <typename Out, int LP>
static hipError_t launch_split(const ScanArgs &sa, const NoisyArgs &na, hipStream_t s)
{
    typedef Fused<Out, 128, LP, true> K2;
    typedef Serve<Out, 128, LP, false, false> K3;
    auto k2 = bdgdn_k2_scan_states_kernel<Out, LP>;
    auto k3 = bdgdn_k3_noisy_kernel<Out, LP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(k2), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  K2::BYTES);
    });
    if (err != hipSuccess) return err;
    const int grid = chain_grid(sa);
    hipLaunchKernelGGL(k2, dim3(grid), dim3(K2::kThreads), K2::BYTES, s, sa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k3, dim3((unsigned)(na.total_blocks * na.h_v)), dim3(K3::kThreads), K3::BYTES, s, na);
    return hipGetLastError();
}

// The clean scan alone, writing the seed state of every block (what the backward and the
// noisy views start from) as SeedT; the clean outputs go to sa.o, of type Out (not with
// STATES: the backward's recomputation).
template <typename Out, typename SeedT, bool STATES = false>
static hipError_t scan_states(int lp, const ScanArgs &sa, hipStream_t s)
{
    auto run = [&](auto k2, int bytes) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void *>(k2),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (err != hipSuccess) return err;
        const int grid = chain_grid(sa);
        hipLaunchKernelGGL(k2, dim3(grid), dim3(768), bytes, s, sa);
        return hipGetLastError();
    };
    return lp == 16 ? run(bdgdn_k2_scan_states_kernel<Out, 16, SeedT, STATES>,
                          Fused<Out, 128, 16, true, true, SeedT, STATES>::BYTES)
                    : run(bdgdn_k2_scan_states_kernel<Out, 32, SeedT, STATES>,
                          Fused<Out, 128, 32, true, true, SeedT, STATES>::BYTES);
}

hipError_t launch_scan_states(int lp, bool f32_out, bool f16_seeds, const ScanArgs &sa, hipStream_t s)
{
    if ((lp != 16 && lp != 32) || sa.n_vt * 32 != sa.dv || !sa.bs) return hipErrorInvalidValue;
    if (f16_seeds)   // the backward's recomputation: seeds only
        return f32_out ? scan_states<float, _Float16, true>(lp, sa, s) : scan_states<__bf16, _Float16, true>(lp, sa, s);
    return f32_out ? scan_states<float, float>(lp, sa, s) : scan_states<__bf16, float>(lp, sa, s);
}

// The noisy-block pass alone (every block of one noisy stream from the seeds in na.bs).
hipError_t launch_noisy_blocks(int lp, bool f32_out, const NoisyArgs &na, hipStream_t s)
{
    if (lp != 16 && lp != 32) return hipErrorInvalidValue;
    if (na.total_blocks * na.h_v == 0) return hipSuccess;
    auto run = [&](auto k3, int bytes) {
        hipLaunchKernelGGL(k3, dim3((unsigned)(na.total_blocks * na.h_v)), dim3(256), bytes, s, na);
        return hipGetLastError();
    };
    if (f32_out)
        return lp == 16 ? run(bdgdn_k3_noisy_kernel<float, 16>, Serve<float, 128, 16, false, false>::BYTES)
                        : run(bdgdn_k3_noisy_kernel<float, 32>, Serve<float, 128, 32, false, false>::BYTES);
    return lp == 16 ? run(bdgdn_k3_noisy_kernel<__bf16, 16>, Serve<__bf16, 128, 16, false, false>::BYTES)
                    : run(bdgdn_k3_noisy_kernel<__bf16, 32>, Serve<__bf16, 128, 32, false, false>::BYTES);
}

bool split_supported(Types ty, int dk, int dv, int lp)
{
    return ty != Types::F32 && dk == 128 && dv == 128 && (lp == 16 || lp == 32);
}

hipError_t launch_fwd_split(Types ty, int lp, const ScanArgs &sa, const NoisyArgs &na, hipStream_t s)
{
    if (!split_supported(ty, 128, sa.dv, lp) || sa.n_vt * 32 != sa.dv || !sa.bs) return hipErrorInvalidValue;
    if (ty == Types::BF16_IN_F32_OUT)
        return lp == 16 ? launch_split<float, 16>(sa, na, s) : launch_split<float, 32>(sa, na, s);
    return lp == 16 ? launch_split<__bf16, 16>(sa, na, s) : launch_split<__bf16, 32>(sa, na, s);
}

}  // namespace bdgdn
