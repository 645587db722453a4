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
// Tile 64 rows x 64 columns, 4 waves as 2 x 2, each 32 x 32 = 2 x 2 MFMA
// blocks of 16 x 16.  K runs in chunks of 32: the next chunk's operands are
// loaded into registers while the current one is multiplied out of LDS.  The
// weight is the MFMA's A operand (a lane's four results are four consecutive
// output columns of one row), the activation row the B operand.

template <bool BF16, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmParams p)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    constexpr int BM = 64, BN = 64, KC = 32;
    constexpr int LD = KC + (BF16 ? 8 : 4);          // padded LDS row: conflict-free 16-byte reads
    constexpr int VE = 16 / (int)sizeof(T);          // elements per 16-byte vector
    constexpr int VPR = KC / VE;                     // vectors per tile row
    constexpr int NV = BM * VPR / 256;               // vectors per thread per operand
    __shared__ __attribute__((aligned(16))) T As[BM * LD];
    __shared__ __attribute__((aligned(16))) T Bs[BN * LD];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const T* A = (const T*)p.A;
    const T* W = (const T*)p.W;

    u32x4 ra[NV], rb[NV];
    auto gload = [&](int k0) {
#pragma unroll
        for (int v = 0; v < NV; v++) {
            const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
            const int row = m0 + r, col = n0 + r;
            ra[v] = row < p.M ? *(const u32x4*)(A + (size_t)row * p.K + k0 + kv) : u32x4{0, 0, 0, 0};
            rb[v] = col < p.N ? *(const u32x4*)(W + (size_t)col * p.K + k0 + kv) : u32x4{0, 0, 0, 0};
        }
    };
    auto lstore = [&]() {
#pragma unroll
        for (int v = 0; v < NV; v++) {
            const int idx = tid + 256 * v, r = idx / VPR, kv = (idx % VPR) * VE;
            *(u32x4*)(As + r * LD + kv) = ra[v];
            *(u32x4*)(Bs + r * LD + kv) = rb[v];
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int l16 = lane & 15, g = lane >> 4;
    const int nk = p.K / KC;
    gload(0);
    for (int kc = 0; kc < nk; kc++) {
        lstore();
        __syncthreads();
        if (kc + 1 < nk) gload((kc + 1) * KC);
        if constexpr (BF16) {
            bf16x8_t wf[2], xf[2];
#pragma unroll
            for (int i = 0; i < 2; i++) wf[i] = *(const bf16x8_t*)(Bs + (wn * 32 + 16 * i + l16) * LD + 8 * g);
#pragma unroll
            for (int j = 0; j < 2; j++) xf[j] = *(const bf16x8_t*)(As + (wm * 32 + 16 * j + l16) * LD + 8 * g);
#pragma unroll
            for (int i = 0; i < 2; i++)
#pragma unroll
                for (int j = 0; j < 2; j++) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[i], xf[j], acc[i][j], 0, 0, 0);
        } else {
#pragma unroll
            for (int s = 0; s < 2; s++) {
                f32x4 wf[2], xf[2];
#pragma unroll
                for (int i = 0; i < 2; i++) wf[i] = *(const f32x4*)(Bs + (wn * 32 + 16 * i + l16) * LD + 16 * s + 4 * g);
#pragma unroll
                for (int j = 0; j < 2; j++) xf[j] = *(const f32x4*)(As + (wm * 32 + 16 * j + l16) * LD + 16 * s + 4 * g);
#pragma unroll
                for (int q = 0; q < 4; q++)
#pragma unroll
                    for (int i = 0; i < 2; i++)
#pragma unroll
                        for (int j = 0; j < 2; j++)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(wf[i][q], xf[j][q], acc[i][j], 0, 0, 0);
            }
        }
        __syncthreads();
    }

    // acc[i][j][r]: row m0 + wm*32 + 16 j + l16, column n0 + wn*32 + 16 i + 4 g + r
#pragma unroll
    for (int i = 0; i < 2; i++) {
        const int col = n0 + wn * 32 + 16 * i + 4 * g;
        if (col >= p.N) continue;
        const f32x4 bias = *(const f32x4*)(p.bias + col);
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const int row = m0 + wm * 32 + 16 * j + l16;
            if (row >= p.M) continue;
            const f32x4 y = acc[i][j] + bias;
            if constexpr (EPI == E_H) {
                *(f32x4*)(p.h + (size_t)row * p.N + col) = y;
            } else if constexpr (EPI == E_RES) {
                float* hp = p.h + (size_t)row * p.N + col;
                const f32x4 gt = *(const f32x4*)(p.gate + col);
                f32x4 hv = *(const f32x4*)hp;
#pragma unroll
                for (int r = 0; r < 4; r++) hv[r] = hv[r] + gt[r] * y[r];
                *(f32x4*)hp = hv;
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
                    const size_t region =
                        (size_t)b * p.carry.stream_stride +
                        ((size_t)((c * 2 + (part - 1)) * p.heads + hd)) * p.carry.Fr * 64;
                    if (part == 1) {
                        store4<BF16>(p.carry.base, region + (size_t)frame * 64 + d, y);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; r++)
                            store1<BF16>(p.carry.base, region + (size_t)(d + r) * p.carry.Fr + frame, y[r]);
                    }
                }
            }
        }
    }
}

hipError_t launch_gemm(const GemmParams& p, int epi, int bf16, hipStream_t st)
{
    const dim3 grid((p.N + 63) / 64, (p.M + 63) / 64);
#define DCF_GEMM(B, E)                                                              \
    if (bf16 == B && epi == E) {                                                    \
        hipLaunchKernelGGL((gemm_kernel<B, E>), grid, dim3(256), 0, st, p);         \
        return hipGetLastError();                                                   \
    }
    DCF_GEMM(1, E_H) DCF_GEMM(1, E_QKV) DCF_GEMM(1, E_RES) DCF_GEMM(1, E_GELU) DCF_GEMM(1, E_VEL)
    DCF_GEMM(0, E_H) DCF_GEMM(0, E_QKV) DCF_GEMM(0, E_RES) DCF_GEMM(0, E_GELU) DCF_GEMM(0, E_VEL)
#undef DCF_GEMM
    return hipErrorInvalidValue;
}

// ------------------------------------------------------- modulated LayerNorm
//
// One wave per row: mean, then the centred second moment (two passes over
// the row held in registers), eps 1e-6, then * (1 + scale) + shift.
template <bool BF16>
__global__ __launch_bounds__(256) void lnmod_kernel(const LnParams p)
{
    constexpr int MAXV = 16;   // dim <= 1024
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= p.M) return;
    const int nv = p.dim / 64;
    const float* hr = p.h + (size_t)row * p.dim;
    float v[MAXV];
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < MAXV; k++)
        if (k < nv) {
            v[k] = hr[lane + 64 * k];
            s += v[k];
        }
    const float mean = wave_sum(s) / (float)p.dim;
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < MAXV; k++)
        if (k < nv) {
            const float d = v[k] - mean;
            q += d * d;
        }
    const float inv = 1.0f / sqrtf(wave_sum(q) / (float)p.dim + 1e-6f);
#pragma unroll
    for (int k = 0; k < MAXV; k++)
        if (k < nv) {
            const int col = lane + 64 * k;
            store1<BF16>(p.out, (size_t)row * p.dim + col, (v[k] - mean) * inv * (1.0f + p.scale[col]) + p.shift[col]);
        }
}

hipError_t launch_lnmod(const LnParams& p, int bf16, hipStream_t st)
{
    const dim3 grid((p.M + 3) / 4);
    if (bf16) hipLaunchKernelGGL((lnmod_kernel<true>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((lnmod_kernel<false>), grid, dim3(256), 0, st, p);
    return hipGetLastError();
}

// --------------------------------------------------------------- attention
//
// Block = (stream, branch, head) x 64 queries; wave w takes queries
// 16 w .. 16 w + 15.  Keys are walked in Eq. carry's logical order -- the
// retained chunks newest first, the prompt, then the call's own frames -- in
// tiles of 32, with a running maximum (online softmax).  Per tile:
//   S^T (keys x queries) = K Q^T        : A = key rows, B = query rows
//   O^T (dims x queries) += V^T P^T     : A = value columns (stored [dim][frame]),
//                                         B = the lane's own probabilities
// In S^T a lane holds keys 4g .. 4g+3 and 16+4g .. 16+4g+3 of the tile for
// query l16 (g = lane / 16); those eight keys, in that order, are the lane's
// K slice of the second product, so P never leaves its registers, and the
// running maximum, sum and rescale of O^T all stay per lane.

template <bool BF16>
__global__ __launch_bounds__(256) void attn_kernel(const AttnParams p)
{
    using T = typename std::conditional<BF16, uint16_t, float>::type;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, g = lane >> 4;
    const int bh = blockIdx.x;
    const int bp = bh / (2 * p.heads), c = (bh / p.heads) & 1, hd = bh % p.heads;
    const int b = p.b0 + bp;
    const int q0 = blockIdx.y * 64 + wave * 16;
    if (q0 >= p.n) return;
    const int fq = q0 + l16;   // this lane's query (rows past n are computed and dropped)

    const T* qp = (const T*)p.q + ((((size_t)bp * 2 + c) * p.heads + hd) * p.Fq + fq) * 64;
    const CarryRef& cr = p.carry;
    const T* Kb = (const T*)cr.base + (size_t)b * cr.stream_stride + ((size_t)((c * 2 + 0) * p.heads + hd)) * cr.Fr * 64;
    const T* Vb = (const T*)cr.base + (size_t)b * cr.stream_stride + ((size_t)((c * 2 + 1) * p.heads + hd)) * cr.Fr * 64;

    // query fragments (B operand of S^T)
    bf16x8_t qb[2];
    f32x4 qf[4];
    if constexpr (BF16) {
#pragma unroll
        for (int s = 0; s < 2; s++) qb[s] = *(const bf16x8_t*)(qp + 32 * s + 8 * g);
    } else {
#pragma unroll
        for (int s = 0; s < 4; s++) qf[s] = *(const f32x4*)(qp + 16 * s + 4 * g);
    }

    float m = -INFINITY, lsum = 0.f;
    f32x4 O[4];
#pragma unroll
    for (int db = 0; db < 4; db++) O[db] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto run = [&](int base, int len) {
        const int last4 = (len - 1) & ~3;
        for (int t0 = 0; t0 < len; t0 += 32) {
            f32x4 st[2];
#pragma unroll
            for (int j = 0; j < 2; j++) {
                st[j] = f32x4{0.f, 0.f, 0.f, 0.f};
                const int key = min(t0 + 16 * j + l16, len - 1);
                const T* kr = Kb + (size_t)(base + key) * 64;
                if constexpr (BF16) {
#pragma unroll
                    for (int s = 0; s < 2; s++)
                        st[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8_t*)(kr + 32 * s + 8 * g), qb[s],
                                                                        st[j], 0, 0, 0);
                } else {
#pragma unroll
                    for (int s = 0; s < 4; s++) {
                        const f32x4 kf = *(const f32x4*)(kr + 16 * s + 4 * g);
#pragma unroll
                        for (int q = 0; q < 4; q++)
                            st[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(kf[q], qf[s][q], st[j], 0, 0, 0);
                    }
                }
            }
            // scores of keys t0 + 16 j + 4 g + r; keys past the segment do not exist
            float mt = -INFINITY;
#pragma unroll
            for (int j = 0; j < 2; j++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const bool live = t0 + 16 * j + 4 * g + r < len;
                    st[j][r] = live ? st[j][r] * 0.125f : -INFINITY;
                    mt = fmaxf(mt, st[j][r]);
                }
            mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float mn = fmaxf(m, mt);
            const float alpha = expf(m - mn);
            m = mn;
            float ps = 0.f;
#pragma unroll
            for (int j = 0; j < 2; j++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    st[j][r] = expf(st[j][r] - mn);
                    ps += st[j][r];
                }
            lsum = lsum * alpha + ps;
#pragma unroll
            for (int db = 0; db < 4; db++) O[db] *= alpha;
            // value groups: keys t0 + 4 g (+16) .. +3, clamped into the segment's storage
            const int ga = min(t0 + 4 * g, last4), gb = min(t0 + 16 + 4 * g, last4);
            if constexpr (BF16) {
                u32x4 pw = {pack2(st[0][0], st[0][1]), pack2(st[0][2], st[0][3]), pack2(st[1][0], st[1][1]),
                            pack2(st[1][2], st[1][3])};
                const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pw);
#pragma unroll
                for (int db = 0; db < 4; db++) {
                    const T* vr = Vb + (size_t)(16 * db + l16) * cr.Fr + base;
                    const u32x2 va = *(const u32x2*)(vr + ga), vb = *(const u32x2*)(vr + gb);
                    const u32x4 vw = {va[0], va[1], vb[0], vb[1]};
                    O[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vw), pf, O[db], 0, 0, 0);
                }
            } else {
#pragma unroll
                for (int db = 0; db < 4; db++) {
                    const T* vr = Vb + (size_t)(16 * db + l16) * cr.Fr + base;
                    const f32x4 va = *(const f32x4*)(vr + ga), vb = *(const f32x4*)(vr + gb);
#pragma unroll
                    for (int q = 0; q < 4; q++) O[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(va[q], st[0][q], O[db], 0, 0, 0);
#pragma unroll
                    for (int q = 0; q < 4; q++) O[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(vb[q], st[1][q], O[db], 0, 0, 0);
                }
            }
        }
    };

    if (!p.prompt) {
        const int64_t hist = cr.hist[b];
        const int nh = hist < cr.R ? (int)hist : cr.R;
        for (int r = 0; r < nh; r++) run(cr.Pr + (int)((hist - 1 - r) % (cr.R + 1)) * cr.Sl, p.f_chunk);
        run(0, cr.plen[b]);
    }
    run(own_base(cr, p.prompt, b), p.n);

    float l1 = lsum + __shfl_xor(lsum, 16, 64);
    l1 = l1 + __shfl_xor(l1, 32, 64);
    const float inv = 1.0f / l1;
    if (fq < p.n) {
        const size_t row = ((size_t)bp * 2 + c) * p.n + fq;
#pragma unroll
        for (int db = 0; db < 4; db++) store4<BF16>(p.o, row * p.dim + hd * 64 + 16 * db + 4 * g, O[db] * inv);
    }
}

hipError_t launch_attn(const AttnParams& p, int Bc, int bf16, hipStream_t st)
{
    const dim3 grid(Bc * 2 * p.heads, (p.n + 63) / 64);
    if (bf16) hipLaunchKernelGGL((attn_kernel<true>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((attn_kernel<false>), grid, dim3(256), 0, st, p);
    return hipGetLastError();
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
