// gfx950 kernels of the streaming flow-decoder chunk step.
//
// One estimator evaluation is a chain of launches over the rows of the call
// (both guidance branches of every stream): an MFMA GEMM per Linear layer
// with its elementwise tail fused into the epilogue (bias, GELU, the gated
// residual add, the scatter of keys and values into the carry), a LayerNorm
// with the step's modulation, and an attention kernel that walks the carried
// keys and values in place.  The K order of every product is fixed by the
// layer alone, and rows never interact outside the attention, so a stream's
// result does not depend on the batch or on which other streams share the
// call.
#include <type_traits>

#include "dc_philox.h"
#include "flow_internal.h"

namespace dcf {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

// Two floats -> packed bfloat16 pair (round to nearest even).
__device__ __forceinline__ uint32_t pack2(float lo, float hi)
{
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ uint16_t f2bf1(float v) { return (uint16_t)(pack2(v, 0.0f) & 0xffffu); }

// Store four consecutive values in the operand type.
template <bool BF16> __device__ __forceinline__ void store4(void* base, size_t idx, f32x4 v)
{
    if constexpr (BF16) {
        u32x2 w = {pack2(v[0], v[1]), pack2(v[2], v[3])};
        *(u32x2*)((uint16_t*)base + idx) = w;
    } else {
        *(f32x4*)((float*)base + idx) = v;
    }
}
template <bool BF16> __device__ __forceinline__ void store1(void* base, size_t idx, float v)
{
    if constexpr (BF16) ((uint16_t*)base)[idx] = f2bf1(v);
    else ((float*)base)[idx] = v;
}

__device__ __forceinline__ float gelu_tanh(float v)
{
    const float k0 = 0.7978845608028654f;   // sqrt(2 / pi)
    return 0.5f * v * (1.0f + tanhf(k0 * (v + 0.044715f * v * v * v)));
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Frame where the call's own frames start in stream b's carry regions.
__device__ __forceinline__ int own_base(const CarryRef& c, int prompt, int b)
{
    if (prompt) return 0;
    return c.Pr + (int)(c.hist[b] % (int64_t)(c.R + 1)) * c.Sl;
}

// ------------------------------------------------------------------- GEMM
//
// Both GEMM kernels take the weight as the MFMA's A operand (a lane's four
// results are four consecutive output columns of one row) and the activation
// row as the B operand, and hand every 4-column group of a row to the same
// epilogue.  With a LayerNorm operand (p.ln_h set) the activation is
// LN(h) * (1 + scale) + shift of the fp32 residual stream h, normalised while
// it is staged: mean and variance per row from sums shifted by the row's
// first value, eps 1e-6.

// The epilogue's operands of one 4-column group (bias; for E_RES also the
// gate and the residual row), loaded apart from their use so that a kernel
// can fetch them before its main loop.
struct EpiPre {
    f32x4 bias, gate, h;
};
template <int EPI>
__device__ __forceinline__ EpiPre epi_prefetch(const GemmParams& p, int row, int col)
{
    EpiPre e;
    e.bias = *(const f32x4*)(p.bias + col);
    if constexpr (EPI == E_RES) {
        e.gate = *(const f32x4*)(p.gate + col);
        e.h = *(const f32x4*)(p.h + (size_t)row * p.N + col);
    }
    return e;
}

template <bool BF16, int EPI>
__device__ __forceinline__ void epilogue4(const GemmParams& p, int row, int col, f32x4 acc, const EpiPre& e)
{
    const f32x4 y = acc + e.bias;
    if constexpr (EPI == E_H) {
        *(f32x4*)(p.h + (size_t)row * p.N + col) = y;
    } else if constexpr (EPI == E_RES) {
        f32x4 hv = e.h;
#pragma unroll
        for (int r = 0; r < 4; r++) hv[r] = hv[r] + e.gate[r] * y[r];
        *(f32x4*)(p.h + (size_t)row * p.N + col) = hv;
    } else if constexpr (EPI == E_GELU) {
        f32x4 z;
#pragma unroll
        for (int r = 0; r < 4; r++) z[r] = gelu_tanh(y[r]);
        store4<BF16>(p.out, (size_t)row * p.N + col, z);
    } else if constexpr (EPI == E_VEL) {
        *(f32x4*)((float*)p.out + (size_t)row * p.N + col) = y;
    } else {   // E_QKV
        const int part = col / p.dim, hd = (col % p.dim) >> 6, d = col & 63;
        const int bp = row / (2 * p.n), c = (row / p.n) & 1, f = row % p.n;
        if (part == 0) {
            store4<BF16>(p.q, ((((size_t)bp * 2 + c) * p.heads + hd) * p.Fq + f) * 64 + d, y);
        } else {
            const int b = p.b0 + bp;
            const int frame = own_base(p.carry, p.prompt, b) + f;
            const size_t region = (size_t)b * p.carry.stream_stride +
                                  ((size_t)((c * 2 + (part - 1)) * p.heads + hd)) * p.carry.Fr * 64;
            if (part == 1) {
                store4<BF16>(p.carry.base, region + (size_t)frame * 64 + d, y);
            } else {
#pragma unroll
                for (int r = 0; r < 4; r++) store1<BF16>(p.carry.base, region + (size_t)(d + r) * p.carry.Fr + frame, y[r]);
            }
        }
    }
}

// LayerNorm statistics of rows m0 .. m0 + 255 / TPR of h [M][K] (K <= 512):
// TPR adjacent threads share a row, thread t taking row t / TPR and columns
// [(t % TPR) K / TPR, (t % TPR + 1) K / TPR).  Returns the row's mean and
// 1 / sqrt(var + eps); the thread's values stay in v.  Mean and variance come
// from sums shifted by the row's first value.
struct LnRow {
    float mean, rstd;
};
template <int TPR, int NV>
__device__ __forceinline__ LnRow ln_row_stats(const float* h, int M, int K, int m0, f32x4 (&v)[NV])
{
    const int tid = threadIdx.x, lane = tid & 63, q = tid % TPR;
    const int row = min(m0 + tid / TPR, M - 1);
    const int kq = K / TPR, nv = kq >> 2;
    const f32x4* hr = (const f32x4*)(h + (size_t)row * K + q * kq);
    // every load is issued (clamped into the thread's columns) before any is used
#pragma unroll
    for (int i = 0; i < NV; i++) v[i] = hr[min(i, nv - 1)];
    const float x0 = __shfl(v[0][0], lane & ~(TPR - 1), 64);
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < NV; i++) {
        const float live = i < nv ? 1.0f : 0.0f;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const float d = (v[i][e] - x0) * live;
            s1 += d;
            s2 += d * d;
        }
    }
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) {
        s1 += __shfl_xor(s1, o, 64);
        s2 += __shfl_xor(s2, o, 64);
    }
    const float md = s1 / (float)K;
    const float var = fmaxf(s2 / (float)K - md * md, 0.f);
    return LnRow{x0 + md, 1.0f / sqrtf(var + 1e-6f)};
}

// Tiled GEMM for many rows: 4 waves as 2 x 2, each 16 MB rows x 16 NB
// columns of MFMA blocks, so a block computes 32 MB x 32 NB.  K runs in
// chunks of KC through two LDS buffers: the next chunk is loaded into
// registers while the current one is multiplied, then stored into the other
// buffer; one barrier per chunk.
template <bool BF16, int EPI, int MB, int NB>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmParams p)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    constexpr int BM = 32 * MB, BN = 32 * NB;
    constexpr int KC = (MB * NB <= 4 ? 128 : 64) / (BF16 ? 1 : 2);
    constexpr int LD = KC + (BF16 ? 8 : 4);          // padded LDS row: conflict-free 16-byte reads
    constexpr int VE = 16 / (int)sizeof(T);          // elements per 16-byte vector
    constexpr int VPR = KC / VE;                     // vectors per tile row
    constexpr int NVA = BM * VPR / 256, NVB = BN * VPR / 256;   // vectors per thread per operand
    constexpr int KQ = BF16 ? 32 : 16;               // K of one MFMA step group
    extern __shared__ __align__(16) unsigned char smem[];
    T* As = (T*)smem;                                // [2][BM * LD]
    T* Bs = As + 2 * BM * LD;                        // [2][BN * LD]

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const T* A = (const T*)p.A;
    const T* W = (const T*)p.W;

    u32x4 ra[NVA], rb[NVB];
    const int kfull = p.K / KC;
    auto gload = [&](int kc) {
        if (kc < kfull) {
#pragma unroll
            for (int v = 0; v < NVA; v++) {
                const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
                ra[v] = *(const u32x4*)(A + (size_t)min(m0 + r, p.M - 1) * p.K + kc * KC + kv);
            }
#pragma unroll
            for (int v = 0; v < NVB; v++) {
                const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
                rb[v] = *(const u32x4*)(W + (size_t)min(n0 + r, p.N - 1) * p.K + kc * KC + kv);
            }
        } else {   // a last partial chunk reads zeros past K
#pragma unroll
            for (int v = 0; v < NVA; v++) {
                const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE, k = kc * KC + kv;
                ra[v] = k < p.K ? *(const u32x4*)(A + (size_t)min(m0 + r, p.M - 1) * p.K + k) : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int v = 0; v < NVB; v++) {
                const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE, k = kc * KC + kv;
                rb[v] = k < p.K ? *(const u32x4*)(W + (size_t)min(n0 + r, p.N - 1) * p.K + k) : u32x4{0, 0, 0, 0};
            }
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int v = 0; v < NVA; v++) {
            const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
            *(u32x4*)(As + (size_t)buf * BM * LD + r * LD + kv) = ra[v];
        }
#pragma unroll
        for (int v = 0; v < NVB; v++) {
            const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
            *(u32x4*)(Bs + (size_t)buf * BN * LD + r * LD + kv) = rb[v];
        }
    };

    f32x4 acc[NB][MB];
#pragma unroll
    for (int i = 0; i < NB; i++)
#pragma unroll
        for (int j = 0; j < MB; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int l16 = lane & 15, g = lane >> 4;
    const int nk = (p.K + KC - 1) / KC;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kc = 0; kc < nk; kc++) {
        const int buf = kc & 1;
        if (kc + 1 < nk) gload(kc + 1);
        const T* Ab = As + (size_t)buf * BM * LD;
        const T* Bb = Bs + (size_t)buf * BN * LD;
#pragma unroll
        for (int s = 0; s < KC / KQ; s++) {
            if constexpr (BF16) {
                bf16x8_t wf[NB], xf[MB];
#pragma unroll
                for (int i = 0; i < NB; i++) wf[i] = *(const bf16x8_t*)(Bb + (wn * 16 * NB + 16 * i + l16) * LD + KQ * s + 8 * g);
#pragma unroll
                for (int j = 0; j < MB; j++) xf[j] = *(const bf16x8_t*)(Ab + (wm * 16 * MB + 16 * j + l16) * LD + KQ * s + 8 * g);
#pragma unroll
                for (int i = 0; i < NB; i++)
#pragma unroll
                    for (int j = 0; j < MB; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[i], xf[j], acc[i][j], 0, 0, 0);
            } else {
                f32x4 wf[NB], xf[MB];
#pragma unroll
                for (int i = 0; i < NB; i++) wf[i] = *(const f32x4*)(Bb + (wn * 16 * NB + 16 * i + l16) * LD + KQ * s + 4 * g);
#pragma unroll
                for (int j = 0; j < MB; j++) xf[j] = *(const f32x4*)(Ab + (wm * 16 * MB + 16 * j + l16) * LD + KQ * s + 4 * g);
#pragma unroll
                for (int q = 0; q < 4; q++)
#pragma unroll
                    for (int i = 0; i < NB; i++)
#pragma unroll
                        for (int j = 0; j < MB; j++)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(wf[i][q], xf[j][q], acc[i][j], 0, 0, 0);
            }
        }
        if (kc + 1 < nk) lstore(buf ^ 1);
        __syncthreads();
    }

    // acc[i][j][r]: row m0 + wm*16 MB + 16 j + l16, column n0 + wn*16 NB + 16 i + 4 g + r
#pragma unroll
    for (int i = 0; i < NB; i++) {
        const int col = n0 + wn * 16 * NB + 16 * i + 4 * g;
        if (col >= p.N) continue;
#pragma unroll
        for (int j = 0; j < MB; j++) {
            const int row = m0 + wm * 16 * MB + 16 * j + l16;
            if (row < p.M) epilogue4<BF16, EPI>(p, row, col, acc[i][j], epi_prefetch<EPI>(p, row, col));
        }
    }
}

template <bool BF16, int MB, int NB>
constexpr size_t tiled_lds_bytes()
{
    constexpr int KC = (MB * NB <= 4 ? 128 : 64) / (BF16 ? 1 : 2);
    return (size_t)2 * (32 * MB + 32 * NB) * (KC + (BF16 ? 8 : 4)) * (BF16 ? 2 : 4);
}

// A kernel launched with more than 64 KB of dynamic LDS needs its limit
// raised first, on each device it runs on: `set` caches, per device, the
// largest size already allowed for that kernel (a race between two threads
// only repeats the call).
constexpr int kMaxDevices = 64;
static hipError_t allow_lds(const void* kernel, size_t lds, size_t (&set)[kMaxDevices])
{
    if (lds <= 64 * 1024) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const bool cached = dev >= 0 && dev < kMaxDevices;
    if (cached && lds <= set[dev]) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess && cached) set[dev] = lds;
    return e;
}

template <bool BF16, int EPI, int MB, int NB>
hipError_t launch_tiled(const GemmParams& p, hipStream_t st)
{
    constexpr size_t lds = tiled_lds_bytes<BF16, MB, NB>();
    static size_t set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&gemm_kernel<BF16, EPI, MB, NB>), lds, set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_kernel<BF16, EPI, MB, NB>), dim3((p.N + 32 * NB - 1) / (32 * NB), (p.M + 32 * MB - 1) / (32 * MB)),
                       dim3(256), lds, st, p);
    return hipGetLastError();
}

// Tile size by the number of 64 x 64 tiles the call would have: at least
// DCF_TILE_BIG_BLOCKS -> 128 x 128, at least DCF_TILE_MID_BLOCKS -> 128 rows x
// 64 columns, fewer -> 32 x 32 (more blocks for calls that would not fill the
// machine).
#ifndef DCF_TILE_BIG_BLOCKS
#define DCF_TILE_BIG_BLOCKS 1024
#endif
#ifndef DCF_TILE_MID_BLOCKS
#define DCF_TILE_MID_BLOCKS 256
#endif

template <bool BF16, int EPI>
hipError_t launch_tiled_any(const GemmParams& p, hipStream_t st)
{
    const long small_blocks = (long)((p.N + 63) / 64) * ((p.M + 63) / 64);
    if (small_blocks >= DCF_TILE_BIG_BLOCKS) return launch_tiled<BF16, EPI, 4, 4>(p, st);
    if (small_blocks >= DCF_TILE_MID_BLOCKS) return launch_tiled<BF16, EPI, 4, 2>(p, st);
    return launch_tiled<BF16, EPI, 1, 1>(p, st);
}

// Skinny GEMM for few rows (a call of a handful of streams): block = 16 RB
// rows x 16 NBLK columns, NW waves that split K into contiguous ranges of whole
// MFMA steps; each wave loads its weight and activation fragments for 4
// steps at once, so a block costs few memory round trips.  The weight loads
// of the first batch and the epilogue's operands are issued before anything
// waits.  The partial tiles are summed through LDS in wave order.  With a
// LayerNorm operand the block first normalises its 16 RB rows into LDS
// (operand type, all K).
template <bool BF16, int EPI, bool LN, int NW, int NBLK, int RB>
__global__ __launch_bounds__(64 * NW) void skinny_kernel(const GemmParams p)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    constexpr int KQ = BF16 ? 32 : 16;               // K of one MFMA step group (one 16-byte load per lane)
    constexpr int BATCH = 4;
    constexpr int PAD = BF16 ? 8 : 4;
    constexpr int NPAIR = RB * NBLK;                 // (column block, row block) output tiles of 16 x 16
    constexpr int TPR = 4 * NW / RB;                 // LayerNorm: threads per row
    static_assert(TPR >= 1 && (TPR & (TPR - 1)) == 0 && TPR * 16 * RB == 64 * NW, "skinny shape");
    constexpr int PPW = (NPAIR + NW - 1) / NW;       // tiles each wave finalises
    extern __shared__ __align__(16) unsigned char smem[];
    T* As = (T*)smem;                                 // LN: [16 RB][K + PAD], then scale and shift
    f32x4* red = (f32x4*)smem;                        // after the main loop: [NW waves][NPAIR][64 lanes]

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, g = lane >> 4;
    const int m0 = blockIdx.y * 16 * RB, n0 = blockIdx.x * 16 * NBLK;
    const int LDA = p.K + PAD;
    const T* A = (const T*)p.A;
    const T* W = (const T*)p.W;

    const int ng = p.K / KQ;
    const int q0 = wave * ng / NW, q1 = (wave + 1) * ng / NW;
    int col[NBLK];
#pragma unroll
    for (int j = 0; j < NBLK; j++) col[j] = min(n0 + 16 * j + l16, p.N - 1);
    // the first batch's weight fragments (they do not wait for the LayerNorm)
    u32x4 wf[BATCH][NBLK];
#pragma unroll
    for (int b = 0; b < BATCH; b++)
#pragma unroll
        for (int j = 0; j < NBLK; j++)
            wf[b][j] = *(const u32x4*)(W + (size_t)col[j] * p.K + min(q0 + b, max(q1 - 1, 0)) * KQ + (BF16 ? 8 : 4) * g);
    // the epilogue's operands of the tiles this wave finalises
    EpiPre pre[PPW];
#pragma unroll
    for (int u = 0; u < PPW; u++) {
        const int pp = min(wave + u * NW, NPAIR - 1), j = pp / RB, i = pp % RB;
        pre[u] = epi_prefetch<EPI>(p, min(m0 + 16 * i + l16, p.M - 1), min(n0 + 16 * j + 4 * g, p.N - 4));
    }

    if constexpr (LN) {
        float* ss = (float*)(smem + (size_t)16 * RB * LDA * sizeof(T));
        for (int k4 = tid; k4 < (p.K >> 2); k4 += 64 * NW) {
            ((f32x4*)ss)[k4] = ((const f32x4*)p.ln_scale)[k4];
            ((f32x4*)(ss + p.K))[k4] = ((const f32x4*)p.ln_shift)[k4];
        }
        // TPR threads per row, K / TPR columns each
        f32x4 v[128 / TPR];
        const LnRow st = ln_row_stats<TPR, 128 / TPR>(p.ln_h, p.M, p.K, m0, v);
        __syncthreads();
        const int r = tid / TPR, kq = p.K / TPR, nv = kq >> 2, kb = (tid % TPR) * kq;
#pragma unroll
        for (int i = 0; i < 128 / TPR; i++)
            if (i < nv) {
                const int k = kb + 4 * i;
                const f32x4 sc = *(const f32x4*)(ss + k), sh = *(const f32x4*)(ss + p.K + k);
                f32x4 a;
#pragma unroll
                for (int u = 0; u < 4; u++) a[u] = (v[i][u] - st.mean) * st.rstd * (1.0f + sc[u]) + sh[u];
                store4<BF16>(As, (size_t)r * LDA + k, a);
            }
        __syncthreads();
    }

    int xr[RB];
#pragma unroll
    for (int i = 0; i < RB; i++) xr[i] = min(m0 + 16 * i + l16, p.M - 1);
    f32x4 acc[NBLK][RB];
#pragma unroll
    for (int j = 0; j < NBLK; j++)
#pragma unroll
        for (int i = 0; i < RB; i++) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int q = q0; q < q1; q += BATCH) {
        // all loads of the batch first; a step past the wave's range reloads
        // its last one with a zero weight fragment, so the loop has no branch
        // (its products add exact zeros: the activations are finite)
        u32x4 xf[BATCH][RB];
        if (q != q0) {
#pragma unroll
            for (int b = 0; b < BATCH; b++)
#pragma unroll
                for (int j = 0; j < NBLK; j++)
                    wf[b][j] = *(const u32x4*)(W + (size_t)col[j] * p.K + min(q + b, q1 - 1) * KQ + (BF16 ? 8 : 4) * g);
        }
#pragma unroll
        for (int b = 0; b < BATCH; b++) {
            const int k = min(q + b, q1 - 1) * KQ + (BF16 ? 8 : 4) * g;
#pragma unroll
            for (int i = 0; i < RB; i++) {
                if constexpr (LN) xf[b][i] = *(const u32x4*)(As + (16 * i + l16) * LDA + k);
                else xf[b][i] = *(const u32x4*)(A + (size_t)xr[i] * p.K + k);
            }
        }
#pragma unroll
        for (int b = 0; b < BATCH; b++) {
            const bool live = q + b < q1;
#pragma unroll
            for (int j = 0; j < NBLK; j++) {
                u32x4 w = wf[b][j];
#pragma unroll
                for (int e = 0; e < 4; e++) w[e] = live ? w[e] : 0u;
#pragma unroll
                for (int i = 0; i < RB; i++) {
                    if constexpr (BF16) {
                        acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w),
                                                                            __builtin_bit_cast(bf16x8_t, xf[b][i]),
                                                                            acc[j][i], 0, 0, 0);
                    } else {
                        const f32x4 wv = __builtin_bit_cast(f32x4, w), xv = __builtin_bit_cast(f32x4, xf[b][i]);
#pragma unroll
                        for (int u = 0; u < 4; u++)
                            acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv[u], xv[u], acc[j][i], 0, 0, 0);
                    }
                }
            }
        }
    }
    if constexpr (LN) __syncthreads();   // the LDS tile becomes the reduction buffer
#pragma unroll
    for (int j = 0; j < NBLK; j++)
#pragma unroll
        for (int i = 0; i < RB; i++) red[(wave * NPAIR + RB * j + i) * 64 + lane] = acc[j][i];
    __syncthreads();
    // wave w sums its tiles over the waves, in wave order
#pragma unroll
    for (int u = 0; u < PPW; u++) {
        const int pp = wave + u * NW;
        if (pp >= NPAIR) break;
        f32x4 y = red[pp * 64 + lane];
#pragma unroll
        for (int w = 1; w < NW; w++) y += red[(w * NPAIR + pp) * 64 + lane];
        const int j = pp / RB, i = pp % RB;
        const int row = m0 + 16 * i + l16, c4 = n0 + 16 * j + 4 * g;
        if (row < p.M && c4 < p.N) epilogue4<BF16, EPI>(p, row, c4, y, pre[u]);
    }
}

// ------------------------------------------------------- modulated LayerNorm
//
// For calls of many rows: out = LN(h) * (1 + scale) + shift, one wave per
// row, the row's values in registers (dim <= 512), mean and variance from
// sums shifted by the row's first value, eps 1e-6; the operand of the
// following tiled GEMM.
template <bool BF16>
__global__ __launch_bounds__(256) void lnmod_kernel(const float* h, void* out, const float* shift, const float* scale,
                                                    int M, int dim)
{
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= M) return;
    const int nv = dim >> 6;
    const float* hr = h + (size_t)row * dim;
    float v[8], sc[8], sh[8];
#pragma unroll
    for (int k = 0; k < 8; k++) {
        const int col = lane + 64 * min(k, nv - 1);
        v[k] = hr[col];
        sc[k] = scale[col];
        sh[k] = shift[col];
    }
    const float x0 = __shfl(v[0], 0, 64);
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int k = 0; k < 8; k++) {
        const float d = (v[k] - x0) * (k < nv ? 1.0f : 0.0f);
        s1 += d;
        s2 += d * d;
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    const float md = s1 / (float)dim;
    const float mean = x0 + md;
    const float rs = 1.0f / sqrtf(fmaxf(s2 / (float)dim - md * md, 0.f) + 1e-6f);
#pragma unroll
    for (int k = 0; k < 8; k++)
        if (k < nv) store1<BF16>(out, (size_t)row * dim + lane + 64 * k, (v[k] - mean) * rs * (1.0f + sc[k]) + sh[k]);
}


// Skinny shapes: waves and 16-column blocks per block, by operand kind.
#ifndef DCF_SK_LN_NBLK
#define DCF_SK_LN_NBLK 2
#endif
#ifndef DCF_SK_PLAIN_NBLK
#define DCF_SK_PLAIN_NBLK 1
#endif
#ifndef DCF_SK_BIGK_WAVES
#define DCF_SK_BIGK_WAVES 8
#endif
#ifndef DCF_SK_PLAIN_WAVES
#define DCF_SK_PLAIN_WAVES 4
#endif
#ifndef DCF_SK_LN_WAVES
#define DCF_SK_LN_WAVES 8
#endif
// 16-row blocks per skinny block, by operand kind
#ifndef DCF_SK_LN_RB
#define DCF_SK_LN_RB 1
#endif
#ifndef DCF_SK_PLAIN_RB
#define DCF_SK_PLAIN_RB 1
#endif
constexpr int kSkinnyBigK = 1024;   // K from which the plain skinny GEMM uses DCF_SK_BIGK_WAVES waves

size_t skinny_lds_bytes(const GemmParams& p, int bf16, int nw, int nblk, int rb)
{
    const size_t red = (size_t)nw * rb * nblk * 64 * 16;
    if (!p.ln_h) return red;
    // the normalised tile, then scale and shift
    const size_t a = (size_t)16 * rb * (p.K + (bf16 ? 8 : 4)) * (bf16 ? 2 : 4) + (size_t)2 * p.K * 4;
    return a > red ? a : red;
}

template <bool BF16, int EPI, bool LN, int NW, int NBLK, int RB>
hipError_t launch_skinny(const GemmParams& p, hipStream_t st)
{
    const size_t lds = skinny_lds_bytes(p, BF16, NW, NBLK, RB);
    static size_t set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&skinny_kernel<BF16, EPI, LN, NW, NBLK, RB>), lds, set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((skinny_kernel<BF16, EPI, LN, NW, NBLK, RB>),
                       dim3((p.N + 16 * NBLK - 1) / (16 * NBLK), (p.M + 16 * RB - 1) / (16 * RB)),
                       dim3(64 * NW), lds, st, p);
    return hipGetLastError();
}

template <bool BF16, int EPI, bool LN>
hipError_t launch_one(const GemmParams& p, hipStream_t st)
{
    if (p.M <= kSkinnyRows) {
        if constexpr (LN) {
            // the LayerNorm staging gives each of a row's 4 NW / RB threads a
            // whole number of 4-column vectors; 4 waves suffice for K = 64
            if (p.K % (16 * DCF_SK_LN_WAVES / DCF_SK_LN_RB) == 0)
                return launch_skinny<BF16, EPI, true, DCF_SK_LN_WAVES, DCF_SK_LN_NBLK, DCF_SK_LN_RB>(p, st);
            return launch_skinny<BF16, EPI, true, 4, DCF_SK_LN_NBLK, 1>(p, st);
        }
        else if (p.K >= kSkinnyBigK)
            return launch_skinny<BF16, EPI, false, DCF_SK_BIGK_WAVES, DCF_SK_PLAIN_NBLK, DCF_SK_PLAIN_RB>(p, st);
        else
            return launch_skinny<BF16, EPI, false, DCF_SK_PLAIN_WAVES, DCF_SK_PLAIN_NBLK, DCF_SK_PLAIN_RB>(p, st);
    } else if (LN) {
        // the normalised operand is written once to p.A by its own launch
        hipLaunchKernelGGL((lnmod_kernel<BF16>), dim3((p.M + 3) / 4), dim3(256), 0, st, p.ln_h, const_cast<void*>(p.A),
                           p.ln_shift, p.ln_scale, p.M, p.K);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        GemmParams q = p;
        q.ln_h = nullptr;
        return launch_tiled_any<BF16, EPI>(q, st);
    }
    return launch_tiled_any<BF16, EPI>(p, st);
}

hipError_t launch_gemm(const GemmParams& p, int epi, int bf16, hipStream_t st)
{
    const bool ln = p.ln_h != nullptr;
#define DCF_GEMM(B, E, L)                                     \
    if (bf16 == B && epi == E && ln == L) return launch_one<B, E, L>(p, st);
    // the LayerNorm operand exists for the GEMMs that follow one; every
    // GEMM can take a plain operand
    DCF_GEMM(1, E_H, false) DCF_GEMM(1, E_QKV, true) DCF_GEMM(1, E_QKV, false) DCF_GEMM(1, E_RES, false)
    DCF_GEMM(1, E_GELU, true) DCF_GEMM(1, E_GELU, false) DCF_GEMM(1, E_VEL, true) DCF_GEMM(1, E_VEL, false)
    DCF_GEMM(0, E_H, false) DCF_GEMM(0, E_QKV, true) DCF_GEMM(0, E_QKV, false) DCF_GEMM(0, E_RES, false)
    DCF_GEMM(0, E_GELU, true) DCF_GEMM(0, E_GELU, false) DCF_GEMM(0, E_VEL, true) DCF_GEMM(0, E_VEL, false)
#undef DCF_GEMM
    return hipErrorInvalidValue;
}

// --------------------------------------------------------------- attention
//
// Block = (stream, branch, head) x up to 64 queries, 8 waves.  The keys, in
// Eq. carry's logical order (the retained chunks newest first, the prompt,
// the call's own frames), are cut into tiles of 32 inside each segment; wave
// w takes tiles w, w + 8, ... for all the block's queries (4 groups of 16),
// loading the next tile while it works on the current one, with a running
// maximum per query (online softmax); the waves' partial results are merged
// through LDS in wave order.  Per tile and query group:
//   S^T (keys x queries) = K Q^T        : A = key rows, B = query rows
//   O^T (dims x queries) += V^T P^T     : A = value columns (stored [dim][frame]),
//                                         B = the lane's own probabilities
// In S^T a lane holds keys 4g .. 4g+3 and 16+4g .. 16+4g+3 of the tile for
// query l16 (g = lane / 16); those eight keys, in that order, are the lane's
// K slice of the second product, so P never leaves its registers, and the
// running maximum, sum and rescale of O^T stay per lane.
constexpr int kMaxSegments = 8;
// Two block shapes: 4 query groups (64 queries) over 8 waves when the call
// has enough (stream, branch, head) blocks to fill the device, else one
// query group (16 queries) over 4 waves, which gives a small call four times
// the blocks.  The shape fixes the order of the softmax merge, so results of
// the two shapes differ in rounding only.
constexpr int kAttnLd = 68;   // padded row of the merge buffer (floats)
// Scores in base 2: q.k / sqrt(64) * log2(e), so the softmax's exponentials are
// plain exp2 (the maximum and the merge work in the same units).
constexpr float kScoreLog2 = 0.125f * 1.4426950408889634f;
constexpr int kAttnWideBlocks = 64;   // blocks of 64 queries below which the narrow shape is used

// per wave: the partial O of its block's 16 QG queries, their running maxima and sums
size_t attn_lds_bytes(int nw, int qg) { return (size_t)nw * 16 * qg * (kAttnLd + 2) * 4; }

template <bool BF16, int QG, int NW>
__global__ __launch_bounds__(64 * NW) void attn_kernel(const AttnParams p)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    static_assert((QG == 1 || QG == 2 || QG == 4) && QG <= NW,
                  "16 * QG divides the 64-row query padding; a merge wave per query group");
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int QB = 16 * QG;                        // queries of the block
    float* Os = (float*)smem;                          // [NW waves][QB queries][kAttnLd]
    float* Ms = Os + NW * QB * kAttnLd;                // [NW][QB]
    float* Ls = Ms + NW * QB;                          // [NW][QB]

    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l16 = lane & 15, g = lane >> 4;
    const int bh = blockIdx.x;
    const int bp = bh / (2 * p.heads), c = (bh / p.heads) & 1, hd = bh % p.heads;
    const int b = p.b0 + bp;
    const int qb0 = blockIdx.y * 16 * QG;
    const CarryRef& cr = p.carry;
    const T* Kb = (const T*)cr.base + (size_t)b * cr.stream_stride + ((size_t)((c * 2 + 0) * p.heads + hd)) * cr.Fr * 64;
    const T* Vb = (const T*)cr.base + (size_t)b * cr.stream_stride + ((size_t)((c * 2 + 1) * p.heads + hd)) * cr.Fr * 64;
    const T* qp = (const T*)p.q + (((size_t)bp * 2 + c) * p.heads + hd) * p.Fq * 64;

    // segments (frame base, length, first global tile) in logical order
    int sb[kMaxSegments], sl[kMaxSegments], st0[kMaxSegments + 1], ns = 0;
    if (!p.prompt) {
        const int64_t hist = cr.hist[b];
        const int nh = hist < cr.R ? (int)hist : cr.R;
        for (int r = 0; r < nh; r++) {
            sb[ns] = cr.Pr + (int)((hist - 1 - r) % (cr.R + 1)) * cr.Sl;
            sl[ns++] = p.f_chunk;
        }
        sb[ns] = 0;
        sl[ns++] = cr.plen[b];
    }
    sb[ns] = own_base(cr, p.prompt, b);
    sl[ns++] = p.n;
    st0[0] = 0;
    for (int i = 0; i < ns; i++) st0[i + 1] = st0[i] + ((sl[i] + 31) >> 5);
    const int total = st0[ns];
    auto locate = [&](int t, int& base, int& len, int& t0) {
        int i = 0;
        while (i + 1 < ns && t >= st0[i + 1]) i++;
        base = sb[i];
        len = sl[i];
        t0 = 32 * (t - st0[i]);
    };

    // one tile's operands: keys (two blocks of 16) and the value groups
    struct Tile {
        u32x4 kf[2][4];
        u32x4 va[4], vb[4];
    };
    auto load = [&](int t, Tile& tl) {
        int base, len, t0;
        locate(t, base, len, t0);
        const int last4 = (len - 1) & ~3;
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const T* kr = Kb + (size_t)(base + min(t0 + 16 * j + l16, len - 1)) * 64;
            if constexpr (BF16) {
#pragma unroll
                for (int s2 = 0; s2 < 2; s2++) tl.kf[j][s2] = *(const u32x4*)(kr + 32 * s2 + 8 * g);
            } else {
#pragma unroll
                for (int s4 = 0; s4 < 4; s4++) tl.kf[j][s4] = *(const u32x4*)(kr + 16 * s4 + 4 * g);
            }
        }
        // value groups: keys t0 + 4 g (+16) .. +3, clamped into the segment's storage
        const int ga = min(t0 + 4 * g, last4), gb2 = min(t0 + 16 + 4 * g, last4);
#pragma unroll
        for (int db = 0; db < 4; db++) {
            const T* vr = Vb + (size_t)(16 * db + l16) * cr.Fr + base;
            if constexpr (BF16) {
                const u32x2 x = *(const u32x2*)(vr + ga), y = *(const u32x2*)(vr + gb2);
                tl.va[db] = u32x4{x[0], x[1], y[0], y[1]};
            } else {
                tl.va[db] = *(const u32x4*)(vr + ga);
                tl.vb[db] = *(const u32x4*)(vr + gb2);
            }
        }
    };

    // query fragments of one group of 16 queries (B operand of S^T)
    struct QFrag {
        bf16x8_t b[2];
        f32x4 f[4];
    };
    auto load_q = [&](int qg, QFrag& qfr) {
        const T* qr = qp + (size_t)(qb0 + 16 * qg + l16) * 64;   // rows past n are computed and dropped
        if constexpr (BF16) {
#pragma unroll
            for (int s2 = 0; s2 < 2; s2++) qfr.b[s2] = *(const bf16x8_t*)(qr + 32 * s2 + 8 * g);
        } else {
#pragma unroll
            for (int s4 = 0; s4 < 4; s4++) qfr.f[s4] = *(const f32x4*)(qr + 16 * s4 + 4 * g);
        }
    };
    // one tile for one query group: scores, running maximum and sum, O^T update
    auto step = [&](const Tile& cur, int t0, int len, const QFrag& qfr, float& m, float& lsum, f32x4 (&O)[4]) {
        f32x4 st[2];
#pragma unroll
        for (int j = 0; j < 2; j++) {
            st[j] = f32x4{0.f, 0.f, 0.f, 0.f};
            if constexpr (BF16) {
#pragma unroll
                for (int s2 = 0; s2 < 2; s2++)
                    st[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, cur.kf[j][s2]),
                                                                    qfr.b[s2], st[j], 0, 0, 0);
            } else {
#pragma unroll
                for (int s4 = 0; s4 < 4; s4++) {
                    const f32x4 kv = __builtin_bit_cast(f32x4, cur.kf[j][s4]);
#pragma unroll
                    for (int u = 0; u < 4; u++)
                        st[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(kv[u], qfr.f[s4][u], st[j], 0, 0, 0);
                }
            }
        }
        float mt = -INFINITY;
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const bool live = t0 + 16 * j + 4 * g + r < len;
                st[j][r] = live ? st[j][r] * kScoreLog2 : -INFINITY;
                mt = fmaxf(mt, st[j][r]);
            }
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float mn = fmaxf(m, mt);
        const float alpha = exp2f(m - mn);
        m = mn;
        float ps = 0.f;
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                st[j][r] = exp2f(st[j][r] - mn);
                ps += st[j][r];
            }
        lsum = lsum * alpha + ps;
#pragma unroll
        for (int db = 0; db < 4; db++) O[db] *= alpha;
        if constexpr (BF16) {
            const u32x4 pw = {pack2(st[0][0], st[0][1]), pack2(st[0][2], st[0][3]), pack2(st[1][0], st[1][1]),
                              pack2(st[1][2], st[1][3])};
            const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pw);
#pragma unroll
            for (int db = 0; db < 4; db++)
                O[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, cur.va[db]), pf, O[db], 0, 0, 0);
        } else {
#pragma unroll
            for (int db = 0; db < 4; db++) {
                const f32x4 va = __builtin_bit_cast(f32x4, cur.va[db]), vb = __builtin_bit_cast(f32x4, cur.vb[db]);
#pragma unroll
                for (int u = 0; u < 4; u++) O[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(va[u], st[0][u], O[db], 0, 0, 0);
#pragma unroll
                for (int u = 0; u < 4; u++) O[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(vb[u], st[1][u], O[db], 0, 0, 0);
            }
        }
    };
    // this wave's partial result of one group: O^T lane (l16, g) holds dims 16 db + 4 g + r of query l16
    auto put = [&](int qg, float m, float lsum, const f32x4 (&O)[4]) {
        float l1 = lsum + __shfl_xor(lsum, 16, 64);
        l1 += __shfl_xor(l1, 32, 64);
        const int qq = 16 * qg + l16;
#pragma unroll
        for (int db = 0; db < 4; db++) *(f32x4*)(Os + ((size_t)wave * QB + qq) * kAttnLd + 16 * db + 4 * g) = O[db];
        if (g == 0) {
            Ms[wave * QB + qq] = m;
            Ls[wave * QB + qq] = l1;
        }
    };

#ifndef DCF_ATTN_PREFETCH
#define DCF_ATTN_PREFETCH 1
#endif
#ifndef DCF_ATTN_QG_ROLLED
#define DCF_ATTN_QG_ROLLED 0
#endif
    if constexpr (DCF_ATTN_QG_ROLLED) {
        // one query group at a time over the wave's tiles (the tiles are
        // read once per group, from L1/L2 after the first): a fourth of the code
#pragma unroll 1
        for (int qg = 0; qg < QG; qg++) {
            QFrag qfr;
            load_q(qg, qfr);
            float m = -INFINITY, lsum = 0.f;
            f32x4 O[4];
#pragma unroll
            for (int db = 0; db < 4; db++) O[db] = f32x4{0.f, 0.f, 0.f, 0.f};
            for (int t = wave; t < total; t += NW) {
                Tile cur;
                load(t, cur);
                int base, len, t0;
                locate(t, base, len, t0);
                step(cur, t0, len, qfr, m, lsum, O);
            }
            put(qg, m, lsum, O);
        }
    } else {
        QFrag qfr[QG];
#pragma unroll
        for (int qg = 0; qg < QG; qg++) load_q(qg, qfr[qg]);
        float m[QG], lsum[QG];
        f32x4 O[QG][4];
#pragma unroll
        for (int qg = 0; qg < QG; qg++) {
            m[qg] = -INFINITY;
            lsum[qg] = 0.f;
#pragma unroll
            for (int db = 0; db < 4; db++) O[qg][db] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        auto work = [&](int t, const Tile& cur) {
            int base, len, t0;
            locate(t, base, len, t0);
#pragma unroll
            for (int qg = 0; qg < QG; qg++) step(cur, t0, len, qfr[qg], m[qg], lsum[qg], O[qg]);
        };
        if constexpr (BF16 && DCF_ATTN_PREFETCH) {
            // the next tile (or this one again) is in flight while one is worked on
            Tile cur;
            load(min(wave, total - 1), cur);
            for (int t = wave; t < total; t += NW) {
                Tile nxt;
                load(min(t + NW, total - 1), nxt);
                work(t, cur);
                cur = nxt;
            }
        } else {   // fp32 tiles are twice the registers: one at a time
            for (int t = wave; t < total; t += NW) {
                Tile cur;
                load(t, cur);
                work(t, cur);
            }
        }
#pragma unroll
        for (int qg = 0; qg < QG; qg++) put(qg, m[qg], lsum[qg], O[qg]);
    }
    __syncthreads();
    if (wave >= QG) return;
    // wave w merges queries 16 w .. 16 w + 15 over the waves, in wave order
    const int qq = 16 * wave + l16;
    float mx = Ms[qq];
#pragma unroll
    for (int w = 1; w < NW; w++) mx = fmaxf(mx, Ms[w * QB + qq]);
    float L = 0.f;
    f32x4 acc[4];
#pragma unroll
    for (int db = 0; db < 4; db++) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < NW; w++) {
        const float sc = exp2f(Ms[w * QB + qq] - mx);
        L += sc * Ls[w * QB + qq];
#pragma unroll
        for (int db = 0; db < 4; db++) acc[db] += sc * *(const f32x4*)(Os + ((size_t)w * QB + qq) * kAttnLd + 16 * db + 4 * g);
    }
    const float inv = 1.0f / L;
    const int fq = qb0 + qq;
    if (fq < p.n) {
        const size_t row = ((size_t)bp * 2 + c) * p.n + fq;
#pragma unroll
        for (int db = 0; db < 4; db++) store4<BF16>(p.o, row * p.dim + hd * 64 + 16 * db + 4 * g, acc[db] * inv);
    }
}

template <bool BF16, int QG, int NW>
hipError_t launch_attn_shape(const AttnParams& p, int Bc, hipStream_t st)
{
    const dim3 grid(Bc * 2 * p.heads, (p.n + 16 * QG - 1) / (16 * QG));
    const size_t lds = attn_lds_bytes(NW, QG);
    static size_t set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&attn_kernel<BF16, QG, NW>), lds, set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_kernel<BF16, QG, NW>), grid, dim3(64 * NW), lds, st, p);
    return hipGetLastError();
}

hipError_t launch_attn(const AttnParams& p, int Bc, int bf16, hipStream_t st)
{
    const bool wide = Bc * 2 * p.heads * ((p.n + 63) / 64) >= kAttnWideBlocks;
    if (bf16) return wide ? launch_attn_shape<true, 4, 8>(p, Bc, st) : launch_attn_shape<true, 1, 4>(p, Bc, st);
    return wide ? launch_attn_shape<false, 4, 8>(p, Bc, st) : launch_attn_shape<false, 1, 4>(p, Bc, st);
}

// ------------------------------------------------------ inputs and the solver

// Row (b', c, f) of the input projection's operand: x | mu | spk | cond, the
// last three zero on the unconditional branch.  x is the initial noise:
// frame tau = pos[b] + f, mel pair j draws Philox4x64-10 at (tau, j, 2, 0)
// under key (seed, keys[b]); Box-Muller of its first two words in fp64.
template <bool BF16>
__global__ __launch_bounds__(256) void assemble_kernel(const AssembleParams p)
{
    const int M4 = 4 * p.n_mel;
    const int64_t total = (int64_t)p.Bc * 2 * p.n * M4;
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= total) return;
    const int col = (int)(e % M4);
    const int row = (int)(e / M4);
    const int bp = row / (2 * p.n), c = (row / p.n) & 1, f = row % p.n;
    const int b = p.b0 + bp;
    const int part = col / p.n_mel, mm = col % p.n_mel;
    float v = 0.f;
    if (part == 0) {
        const dc::Philox4 r = dc::philox4x64_10((uint64_t)(p.pos[b] + f), (uint64_t)(mm >> 1), 2, 0, p.seed, p.keys[b]);
        const double rad = sqrt(-2.0 * log(dc::to_u01(r.v[0])));
        const double ang = 2.0 * M_PI * dc::to_u01(r.v[1]);
        v = p.temperature * (float)((mm & 1) ? rad * sin(ang) : rad * cos(ang));
        if (c == 0) p.x[((size_t)bp * p.n + f) * p.n_mel + mm] = v;
    } else if (c == 0) {
        const size_t fi = ((size_t)bp * p.n + f) * p.n_mel + mm;
        v = part == 1 ? p.mu[fi] : part == 2 ? p.spk[(size_t)b * p.n_mel + mm] : (p.cond ? p.cond[fi] : 0.f);
    }
    store1<BF16>(p.xin, (size_t)row * M4 + col, v);
}

hipError_t launch_assemble(const AssembleParams& p, int bf16, hipStream_t st)
{
    const int64_t total = (int64_t)p.Bc * 2 * p.n * 4 * p.n_mel;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (bf16) hipLaunchKernelGGL((assemble_kernel<true>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((assemble_kernel<false>), grid, dim3(256), 0, st, p);
    return hipGetLastError();
}

// x += dt * ((1 + w) v_cond - w v_uncond); the x columns of both branches'
// operand rows follow; the last step writes the mel output instead.
template <bool BF16>
__global__ __launch_bounds__(256) void euler_kernel(const EulerParams p)
{
    const int64_t total = (int64_t)p.Bc * p.n * p.n_mel;
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= total) return;
    const int mm = (int)(e % p.n_mel);
    const int f = (int)((e / p.n_mel) % p.n);
    const int bp = (int)(e / ((int64_t)p.n_mel * p.n));
    const size_t rc = ((size_t)bp * 2 * p.n + f), ru = rc + p.n;
    const float vc = p.v[rc * p.n_mel + mm], vu = p.v[ru * p.n_mel + mm];
    const float x = p.x[e] + p.dt[0] * ((1.0f + p.w) * vc - p.w * vu);
    p.x[e] = x;
    if (p.mel) {
        p.mel[e] = x;
    } else {
        store1<BF16>(p.xin, rc * 4 * p.n_mel + mm, x);
        store1<BF16>(p.xin, ru * 4 * p.n_mel + mm, x);
    }
}

hipError_t launch_euler(const EulerParams& p, int bf16, hipStream_t st)
{
    const int64_t total = (int64_t)p.Bc * p.n * p.n_mel;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (bf16) hipLaunchKernelGGL((euler_kernel<true>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((euler_kernel<false>), grid, dim3(256), 0, st, p);
    return hipGetLastError();
}

// -------------------------------------------------- per-step constants (init)
//
// The modulations depend only on the step's time t_i: one block per step
// computes the time grid, the sinusoidal embedding of 1000 t_i, the time MLP
// and SiLU of its output; a second launch maps that through every block's
// ada layer (one thread per output).
__global__ __launch_bounds__(256) void temb_kernel(const ConstParams p)
{
    __shared__ float e[1024];
    __shared__ float g[1024];
    const int i = blockIdx.x, tid = threadIdx.x;
    const double ti = 1.0 - cos(0.5 * M_PI * (double)i / (double)p.NS);
    if (tid == 0) {
        const double tn = 1.0 - cos(0.5 * M_PI * (double)(i + 1) / (double)p.NS);
        p.t[i] = (float)ti;
        p.dt[i] = (float)(tn - ti);
        if (i == p.NS - 1) p.t[p.NS] = (float)tn;
    }
    const int half = p.t_dim / 2;
    for (int j = tid; j < half; j += 256) {
        const double arg = 1000.0 * ti * exp(-log(10000.0) * (double)j / (double)half);
        e[j] = (float)cos(arg);
        e[half + j] = (float)sin(arg);
    }
    __syncthreads();
    for (int o = tid; o < p.dim; o += 256) {
        float s = p.b1[o];
        for (int k = 0; k < p.t_dim; k++) s += p.W1[(size_t)o * p.t_dim + k] * e[k];
        g[o] = s / (1.0f + expf(-s));
    }
    __syncthreads();
    for (int o = tid; o < p.dim; o += 256) {
        float s = p.b2[o];
        for (int k = 0; k < p.dim; k++) s += p.W2[(size_t)o * p.dim + k] * g[k];
        p.silu_temb[(size_t)i * p.dim + o] = s / (1.0f + expf(-s));
    }
}

__global__ __launch_bounds__(256) void mods_kernel(const ConstParams p)
{
    const int i = blockIdx.y, l = blockIdx.z;   // l == NL: the final layer
    const int outs = l < p.NL ? 6 * p.dim : 2 * p.dim;
    const int o = blockIdx.x * 256 + threadIdx.x;
    if (o >= outs) return;
    const float* W = l < p.NL ? p.ada + (size_t)l * p.ada_stride : p.fada;
    const float* bias = W + (size_t)outs * p.dim;
    const float* s = p.silu_temb + (size_t)i * p.dim;
    float acc = bias[o];
    for (int k = 0; k < p.dim; k++) acc += W[(size_t)o * p.dim + k] * s[k];
    if (l < p.NL) p.mods[((size_t)i * p.NL + l) * 6 * p.dim + o] = acc;
    else p.fmods[(size_t)i * 2 * p.dim + o] = acc;
}

hipError_t launch_consts(const ConstParams& p, hipStream_t st)
{
    hipLaunchKernelGGL(temb_kernel, dim3(p.NS), dim3(256), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(mods_kernel, dim3((6 * p.dim + 255) / 256, p.NS, p.NL + 1), dim3(256), 0, st, p);
    return hipGetLastError();
}

// ------------------------------------------------------------ stream state

__global__ void advance_kernel(int64_t* hist, int64_t* pos, int* plen, int mode, int b, int P, int B, int f_chunk)
{
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (mode == 0) {
        if (t == 0) {
            hist[b] = 0;
            pos[b] = 0;
            plen[b] = 0;
        }
    } else if (mode == 1) {
        if (t == 0) {
            pos[b] = P;
            plen[b] = P;
        }
    } else if (t < B) {
        hist[t] += 1;
        pos[t] += f_chunk;
    }
}

hipError_t launch_advance(int64_t* hist, int64_t* pos, int* plen, int mode, int b, int P, int B, int f_chunk,
                          hipStream_t st)
{
    hipLaunchKernelGGL(advance_kernel, dim3((B + 255) / 256), dim3(256), 0, st, hist, pos, plen, mode, b, P, B,
                       f_chunk);
    return hipGetLastError();
}

// Carry of (stream b, branch c, kv) at the step and block of cr.base in
// logical order: frames [0, nh * f_chunk) the retained chunks newest first,
// then the prompt; out [frames][heads * 64] fp32.
template <bool BF16>
__global__ __launch_bounds__(256) void gather_kernel(const CarryRef cr, int b, int c, int kv, int heads, int f_chunk,
                                                     int frames, float* out)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int dim = heads * 64;
    if (e >= (int64_t)frames * dim) return;
    const int f = (int)(e / dim), col = (int)(e % dim), hd = col >> 6, d = col & 63;
    const int64_t hist = cr.hist[b];
    const int nh = hist < cr.R ? (int)hist : cr.R;
    int phys;
    if (f < nh * f_chunk) {
        const int r = f / f_chunk;
        phys = cr.Pr + (int)((hist - 1 - r) % (cr.R + 1)) * cr.Sl + f % f_chunk;
    } else {
        phys = f - nh * f_chunk;
    }
    const T* reg = (const T*)cr.base + (size_t)b * cr.stream_stride + ((size_t)((c * 2 + kv) * heads + hd)) * cr.Fr * 64;
    const T v = kv == 0 ? reg[(size_t)phys * 64 + d] : reg[(size_t)d * cr.Fr + phys];
    if constexpr (BF16) out[e] = bf2f(v);
    else out[e] = v;
}

hipError_t launch_carry_gather(const CarryRef& c, int b, int branch, int kv, int heads, int bf16, int frames,
                               int f_chunk, float* out, hipStream_t st)
{
    const int64_t total = (int64_t)frames * heads * 64;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (bf16) hipLaunchKernelGGL((gather_kernel<true>), grid, dim3(256), 0, st, c, b, branch, kv, heads, f_chunk, frames, out);
    else hipLaunchKernelGGL((gather_kernel<false>), grid, dim3(256), 0, st, c, b, branch, kv, heads, f_chunk, frames, out);
    return hipGetLastError();
}

}  // namespace dcf
