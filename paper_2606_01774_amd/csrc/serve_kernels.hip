// serve_kernels.hip -- Diffusion-Trust serving passes over a pool of cached fp32
// states: the denoise pass (block-end readout, the state is only read) and the
// token-causal commit pass (the state is advanced and written back in place).
// bf16 inputs with d_k = d_v = 128 and blocks of up to 32 positions run the streaming
// kernels of serve.hpp (one workgroup per (request, v-head), state straight to
// registers); every other shape runs the general engine, one workgroup per (request,
// v-head, d_v tile).  Each workgroup reads its state tile once.
#include <mutex>

#include "engine.hpp"
#include "kernels.hpp"
#include "serve.hpp"

namespace bdgdn {

#ifndef BDGDN_SERVE_BV
#define BDGDN_SERVE_BV 64
#endif
#ifndef BDGDN_SERVE_NW
#define BDGDN_SERVE_NW 8
#endif
constexpr int kServeBV = BDGDN_SERVE_BV;  // d_v columns per workgroup
constexpr int kServeNW = BDGDN_SERVE_NW;  // waves per workgroup
constexpr int kServeThreads = 64 * kServeNW;

template <typename In, typename Op, typename Out, int DK, int BV, int LP, bool CL, bool CO, bool NZ>
__device__ __forceinline__ void serve_body(const ServeArgs &a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Engine<In, Op, Out, DK, BV, LP, CL, CO, NZ, kServeNW> Eng;
    const int id = blockIdx.x;
    const int unit = id / a.n_vt, vt = id % a.n_vt;
    const int r = unit / a.h_v, h = unit % a.h_v;
    const int sl = a.slot ? a.slot[r] : r;
    const int hq = h / (a.h_v / a.h_qk);
    const int v0 = vt * BV;
    Eng eng(smem);
    f32x4 S[Eng::NSW];
    float *state = a.pool + ((long)sl * a.h_v + h) * DK * a.dv + v0;
    eng.load_state(S, state, a.dv);
    eng.write_st(S);
    __syncthreads();
    typename Eng::IO io;
    io.qk_stride = (long)a.h_qk * DK;
    io.v_stride = (long)a.h_v * a.dv;
    io.gate_stride = a.h_v;
    const long row0 = (long)r * a.L;
    const long qk_off = (row0 * a.h_qk + hq) * DK;
    const long v_off = (row0 * a.h_v + h) * a.dv + v0;
    const long g_off = row0 * a.h_v + h;
    const In *q = static_cast<const In *>(a.q) + qk_off;
    const In *k = static_cast<const In *>(a.k) + qk_off;
    const In *v = static_cast<const In *>(a.v) + v_off;
    Out *o = a.o ? static_cast<Out *>(a.o) + v_off : nullptr;
    io.k = k; io.q = q; io.v = v;
    io.kn = k; io.qn = q; io.vn = v;
    io.g = a.g + g_off; io.beta = a.beta + g_off;
    io.gn = a.g + g_off; io.betan = a.beta + g_off;
    io.o = o; io.on = o;
    io.nvalid = a.L;
    typename Eng::Fetched f;
    eng.fetch(io, f);
    eng.step(io, false, io, f, S, a.scale);
    if (CL) eng.store_state(S, state, a.dv);
}

template <typename In, typename Op, typename Out, int DK, int BV, int LP>
__global__ void __launch_bounds__(kServeThreads) bdgdn_denoise_kernel(ServeArgs a)
{
    serve_body<In, Op, Out, DK, BV, LP, false, false, true>(a);
}

template <typename In, typename Op, typename Out, int DK, int BV, int LP, bool CO>
__global__ void __launch_bounds__(kServeThreads) bdgdn_commit_kernel(ServeArgs a)
{
    serve_body<In, Op, Out, DK, BV, LP, true, CO, false>(a);
}

// ---- streaming kernels (serve.hpp)
template <typename Out, int LP, bool COMMIT, bool CO, bool REC = false>
__device__ __forceinline__ void stream_body(const ServeArgs &a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    typedef Serve<Out, 128, LP, COMMIT, CO, REC> K;
    typedef typename K::In In;
    const int unit = blockIdx.x;
    const int r = unit / a.h_v, h = unit % a.h_v;
    const int sl = a.slot ? a.slot[r] : r;
    const int hq = h / (a.h_v / a.h_qk);
    typename K::Unit u;
    const long row0 = (long)r * a.L;
    const long qk_off = (row0 * a.h_qk + hq) * 128;
    const long v_off = (row0 * a.h_v + h) * 128;
    u.k = static_cast<const In *>(a.k) + qk_off;
    u.q = static_cast<const In *>(a.q) + qk_off;
    u.v = static_cast<const In *>(a.v) + v_off;
    u.g = a.g + row0 * a.h_v + h;
    u.beta = a.beta + row0 * a.h_v + h;
    u.state = a.pool + ((long)sl * a.h_v + h) * 128 * 128;
    u.o = a.o ? static_cast<Out *>(a.o) + v_off : nullptr;
    u.qks = a.h_qk * 128;
    u.vst = a.h_v * 128;
    u.gst = a.h_v;
    u.nvalid = a.L;
    u.scale = a.scale;
    u.states = REC ? a.states + ((long)r * a.n_rec * a.h_v + h) * 128 * 128 : nullptr;
    u.n_rec = REC ? a.n_rec : 0;
    u.rec_step = (long)a.h_v * 128 * 128;
    K k(smem);
    k.run(u);
}

template <typename Out, int LP>
__global__ void __launch_bounds__(256) bdgdn_k4_denoise_kernel(ServeArgs a)
{
    stream_body<Out, LP, false, false>(a);
}

template <typename Out, int LP, bool CO>
__global__ void __launch_bounds__(256) bdgdn_k4_commit_kernel(ServeArgs a)
{
    stream_body<Out, LP, true, CO>(a);
}

template <typename Out, int LP, bool CO>
__global__ void __launch_bounds__(256) bdgdn_k4_commit_record_kernel(ServeArgs a)
{
    stream_body<Out, LP, true, CO, true>(a);
}

// The accept step of the verify-state cache: one workgroup per (request, v-head) copies
// the recorded state at the request's accepted offset into its pool slot (16-byte
// accesses, each thread strided by the workgroup); offsets at or past n_rec (the pool
// already holds the pass's final state) and negative ones leave the slot untouched.
__global__ void __launch_bounds__(256) bdgdn_accept_states_kernel(ServeArgs a, int ssz4)
{
    const int r = blockIdx.x / a.h_v, h = blockIdx.x % a.h_v;
    const int acc = a.accept[r];
    if (acc < 0 || acc >= a.n_rec) return;
    const int sl = a.slot ? a.slot[r] : r;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(a.states) + (((long)r * a.n_rec + acc) * a.h_v + h) * ssz4;
    f32x4 *dst = reinterpret_cast<f32x4 *>(a.pool) + ((long)sl * a.h_v + h) * ssz4;
    for (int i = threadIdx.x; i < ssz4; i += 256) dst[i] = src[i];
}

template <typename K>
static hipError_t set_lds(K kern, int bytes, std::once_flag &once, hipError_t &err)
{
    std::call_once(once, [&] {
        err = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    });
    return err;
}

template <typename In, typename Op, typename Out, int DK, int LP>
static hipError_t launch_dn(const ServeArgs &a, hipStream_t s)
{
    typedef Layout<Op, DK, kServeBV, LP, false, false, true> Ly;
    static_assert(Ly::BYTES <= 160 * 1024, "LDS budget");
    auto kern = bdgdn_denoise_kernel<In, Op, Out, DK, kServeBV, LP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    if (set_lds(kern, Ly::BYTES, once, err) != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(a.R * a.h_v * a.n_vt), dim3(kServeThreads), Ly::BYTES, s, a);
    return hipGetLastError();
}

template <typename In, typename Op, typename Out, int DK, int LP, bool CO>
static hipError_t launch_cm1(const ServeArgs &a, hipStream_t s)
{
    typedef Layout<Op, DK, kServeBV, LP, true, CO, false> Ly;
    static_assert(Ly::BYTES <= 160 * 1024, "LDS budget");
    auto kern = bdgdn_commit_kernel<In, Op, Out, DK, kServeBV, LP, CO>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    if (set_lds(kern, Ly::BYTES, once, err) != hipSuccess) return err;
    hipLaunchKernelGGL(kern, dim3(a.R * a.h_v * a.n_vt), dim3(kServeThreads), Ly::BYTES, s, a);
    return hipGetLastError();
}

template <typename In, typename Op, typename Out, int DK, int LP>
static hipError_t launch_cm(bool with_o, const ServeArgs &a, hipStream_t s)
{
    return with_o ? launch_cm1<In, Op, Out, DK, LP, true>(a, s) : launch_cm1<In, Op, Out, DK, LP, false>(a, s);
}

#define BDGDN_SERVE_DISPATCH(CALL)                                                       \
    switch (ty) {                                                                        \
    case Types::BF16_IN_F32_OUT:                                                         \
        BDGDN_LPS(CALL, __bf16, _Float16, float, 64) BDGDN_LPS(CALL, __bf16, _Float16, float, 128) \
        break;                                                                           \
    case Types::BF16_IN_BF16_OUT:                                                        \
        BDGDN_LPS(CALL, __bf16, _Float16, __bf16, 64) BDGDN_LPS(CALL, __bf16, _Float16, __bf16, 128) \
        break;                                                                           \
    case Types::F32:                                                                     \
        BDGDN_ONE(CALL, float, float, float, 64, 16) BDGDN_ONE(CALL, float, float, float, 64, 32) \
        BDGDN_ONE(CALL, float, float, float, 128, 16) BDGDN_ONE(CALL, float, float, float, 128, 32) \
        break;                                                                           \
    }
#define BDGDN_LPS(CALL, IN, OP, OUT, DK) \
    BDGDN_ONE(CALL, IN, OP, OUT, DK, 16) BDGDN_ONE(CALL, IN, OP, OUT, DK, 32) BDGDN_ONE(CALL, IN, OP, OUT, DK, 64)

int serve_tile_v() { return kServeBV; }

static bool stream_ok(Types ty, int dk, int lp, const ServeArgs &a)
{
    return ty != Types::F32 && dk == 128 && a.dv == 128 && (lp == 16 || lp == 32);
}

template <typename Out, int LP, bool COMMIT, bool CO>
static hipError_t launch_stream(const ServeArgs &a, hipStream_t s)
{
    typedef Serve<Out, 128, LP, COMMIT, CO> K;
    static_assert(K::BYTES <= 64 * 1024, "LDS budget");
    void (*kern)(ServeArgs);
    if constexpr (COMMIT)
        kern = bdgdn_k4_commit_kernel<Out, LP, CO>;
    else
        kern = bdgdn_k4_denoise_kernel<Out, LP>;
    hipLaunchKernelGGL(kern, dim3(a.R * a.h_v), dim3(K::kThreads), K::BYTES, s, a);
    return hipGetLastError();
}

template <typename Out, int LP, bool CO>
static hipError_t launch_record(const ServeArgs &a, hipStream_t s)
{
    typedef Serve<Out, 128, LP, true, CO, true> K;
    hipLaunchKernelGGL((bdgdn_k4_commit_record_kernel<Out, LP, CO>), dim3(a.R * a.h_v), dim3(K::kThreads), K::BYTES,
                       s, a);
    return hipGetLastError();
}

bool record_supported(Types ty, int dk, int dv, int lp)
{
    return ty != Types::F32 && dk == 128 && dv == 128 && (lp == 16 || lp == 32);
}

hipError_t launch_commit_record(Types ty, int lp, bool with_o, const ServeArgs &a, hipStream_t s)
{
    if (!record_supported(ty, 128, a.dv, lp) || !a.states || a.n_rec < 1 || a.n_rec > a.L) return hipErrorInvalidValue;
#define BDGDN_REC(OUT) \
    return with_o ? (lp == 16 ? launch_record<OUT, 16, true>(a, s) : launch_record<OUT, 32, true>(a, s)) \
                  : (lp == 16 ? launch_record<OUT, 16, false>(a, s) : launch_record<OUT, 32, false>(a, s));
    if (ty == Types::BF16_IN_F32_OUT) {
        BDGDN_REC(float)
    }
    BDGDN_REC(__bf16)
#undef BDGDN_REC
}

hipError_t launch_accept_states(const ServeArgs &a, int dk, hipStream_t s)
{
    if (!a.states || !a.accept || a.n_rec < 1 || (dk * a.dv) % 4) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bdgdn_accept_states_kernel, dim3(a.R * a.h_v), dim3(256), 0, s, a, dk * a.dv / 4);
    return hipGetLastError();
}

template <bool COMMIT, bool CO>
static hipError_t dispatch_stream(Types ty, int lp, const ServeArgs &a, hipStream_t s)
{
    if (ty == Types::BF16_IN_F32_OUT)
        return lp == 16 ? launch_stream<float, 16, COMMIT, CO>(a, s) : launch_stream<float, 32, COMMIT, CO>(a, s);
    return lp == 16 ? launch_stream<__bf16, 16, COMMIT, CO>(a, s) : launch_stream<__bf16, 32, COMMIT, CO>(a, s);
}

hipError_t launch_denoise(Types ty, int dk, int lp, const ServeArgs &a, hipStream_t s)
{
    if (stream_ok(ty, dk, lp, a)) return dispatch_stream<false, false>(ty, lp, a, s);
    if (a.dv % kServeBV || a.n_vt * kServeBV != a.dv) return hipErrorInvalidValue;
#define BDGDN_ONE(CALL, IN, OP, OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_dn<IN, OP, OUT, DK, LP>(a, s);
    BDGDN_SERVE_DISPATCH(0)
#undef BDGDN_ONE
    return hipErrorInvalidValue;
}

hipError_t launch_commit(Types ty, int dk, int lp, bool with_o, const ServeArgs &a, hipStream_t s)
{
    if (stream_ok(ty, dk, lp, a))
        return with_o ? dispatch_stream<true, true>(ty, lp, a, s) : dispatch_stream<true, false>(ty, lp, a, s);
    if (a.dv % kServeBV || a.n_vt * kServeBV != a.dv) return hipErrorInvalidValue;
#define BDGDN_ONE(CALL, IN, OP, OUT, DK, LP) \
    if (dk == DK && lp == LP) return launch_cm<IN, OP, OUT, DK, LP>(with_o, a, s);
    BDGDN_SERVE_DISPATCH(0)
#undef BDGDN_ONE
    return hipErrorInvalidValue;
}

#undef BDGDN_LPS
#undef BDGDN_SERVE_DISPATCH

}  // namespace bdgdn
