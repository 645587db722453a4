// gfx950 kernels of the streaming Token2Wav decode step.
//
// Every causal layer is one implicit-GEMM launch (conv_kernel): a block owns a
// tile of BM consecutive frames of one stream and BN output columns, stages
// the operand rows it needs -- the tile plus the (k-1)*d frames of left
// context, read through the input ring, so the carried context of the
// previous call and the frames of this call are the same loads -- into LDS
// once per channel block, and walks the taps as row offsets into that LDS
// tile.  Weights stream from L2 in MFMA fragment order.  The K order (channel
// block, tap, channel) depends only on the layer, never on the tile shape,
// the call size or the batch, and MFMA accumulation is per output element, so
// a frame's value is the same wherever it falls in a tile: chunked and
// offline decoding agree bit for bit (Design, Definition 2; Proposition 1's
// premise that replay issues identical kernels over identical shapes).
#include "dc_internal.h"

namespace dc {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// ------------------------------------------------------------------ helpers

// float -> bfloat16 bits, round to nearest, ties to even (NaN kept quiet).
__device__ __forceinline__ uint32_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (u >> 16) | ((u & 0x007fffffu) ? 0x40u : 0u);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ float lrelu(float v, float s) { return v >= 0.0f ? v : v * s; }

__device__ __forceinline__ int64_t ring_slot(int64_t tau, int64_t R)
{
    int64_t s = tau % R;
    return s < 0 ? s + R : s;
}

// ----------------------------------------------------- operand type traits

template <bool BF16> struct OpT;

// bf16 operands: v_mfma_f32_16x16x32_bf16, lane l holds 8 consecutive K
// values (channels 8*(l/16) .. +7 of a 32-channel chunk) of row/col l%16.
template <> struct OpT<true> {
    using T = uint16_t;
    static constexpr int KQ = 32;   // channels per MFMA step
    static constexpr int PAD = 8;   // LDS row padding (elements)
};

// fp32 operands: v_mfma_f32_16x16x4_f32 four times per 16-channel chunk; in
// step q lane l holds channel 4*(l/16) + q, so one 16-byte load per lane
// feeds four steps.
template <> struct OpT<false> {
    using T = float;
    static constexpr int KQ = 16;
    static constexpr int PAD = 4;
};

// Load 8 channels of one frame as floats (zeros when absent).
__device__ __forceinline__ void load8(const void* base, int elem, size_t off, float v[8])
{
    if (elem == kF32) {
        const f32x4* p = (const f32x4*)((const float*)base + off);
        f32x4 a = p[0], b = p[1];
        v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
        v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
    } else {
        u32x4 a = *(const u32x4*)((const uint16_t*)base + off);
#pragma unroll
        for (int e = 0; e < 4; e++) {
            v[2 * e] = bf2f(a[e] & 0xffffu);
            v[2 * e + 1] = bf2f(a[e] >> 16);
        }
    }
}

__device__ __forceinline__ void store8_lds(uint16_t* dst, const float v[8])
{
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; e++) w[e] = f2bf(v[2 * e]) | (f2bf(v[2 * e + 1]) << 16);
    *(u32x4*)dst = w;
}

__device__ __forceinline__ void store8_lds(float* dst, const float v[8])
{
    f32x4 a = {v[0], v[1], v[2], v[3]}, b = {v[4], v[5], v[6], v[7]};
    *(f32x4*)dst = a;
    *(f32x4*)(dst + 4) = b;
}

// ------------------------------------------------------------ causal conv

template <bool BF16, int BM, int BN, int WGM>
__global__ __launch_bounds__(256) void conv_kernel(ConvParams p)
{
    using Tr = OpT<BF16>;
    using T = typename Tr::T;
    constexpr int WGN = 4 / WGM;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int MB = WM / 16, NB = WN / 16;
    static_assert(WGM * WGN == 4 && MB >= 1 && NB >= 1, "tile shape");

    extern __shared__ __align__(16) unsigned char smem[];
    T* lds = reinterpret_cast<T*>(smem);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WGM, wn = wave / WGM;
    const int b = blockIdx.x / p.tiles_t;
    const int t0 = (blockIdx.x % p.tiles_t) * BM;
    const int n0 = blockIdx.y * BN;
    const int64_t tau0 = p.clock[0] * p.in_fpt;
    const int halo = (p.k - 1) * p.d;
    const int rows = BM + halo;
    const int ldw = p.CB + Tr::PAD;
    const int vpr = p.CB / 8;               // 8-channel vectors per LDS row
    const int kchunks = p.CB / Tr::KQ;

    f32x4 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; i++)
#pragma unroll
        for (int j = 0; j < NB; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int cb = 0; cb < p.n_cb; cb++) {
        __syncthreads();
        // Stage the operand rows [t0 - halo, t0 + BM) of this channel block.
        for (int v = tid; v < rows * vpr; v += 256) {
            const int r = v / vpr, c8 = (v - r * vpr) * 8;
            const int t = t0 - halo + r;
            const int ch = cb * p.CB + c8;
            float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            if (t < p.F && ch < p.in_C) {
                const int64_t slot = ring_slot(tau0 + t, p.in_R);
                load8(p.in, p.in_elem, ((size_t)b * p.in_R + slot) * p.in_C + ch, x);
                if (p.in_act) {
#pragma unroll
                    for (int e = 0; e < 8; e++) x[e] = lrelu(x[e], p.slope);
                }
            }
            store8_lds(lds + r * ldw + c8, x);
        }
        __syncthreads();

        for (int j = 0; j < p.k; j++) {
            const int roff = j * p.d;
            for (int kc = 0; kc < kchunks; kc++) {
                const size_t wbase = ((size_t)(cb * p.k + j) * kchunks + kc) * p.NB16;
                if constexpr (BF16) {
                    bf16x8_t a[MB], w[NB];
#pragma unroll
                    for (int mb = 0; mb < MB; mb++) {
                        const int row = wm * WM + mb * 16 + (lane & 15) + roff;
                        a[mb] = __builtin_bit_cast(bf16x8_t,
                                                   *(const u32x4*)(lds + row * ldw + kc * 32 + (lane >> 4) * 8));
                    }
#pragma unroll
                    for (int nb = 0; nb < NB; nb++) {
                        const int nblk = (n0 + wn * WN) / 16 + nb;
                        u32x4 wv = {0u, 0u, 0u, 0u};
                        if (nblk < p.NB16) wv = ((const u32x4*)p.wp)[(wbase + nblk) * 64 + lane];
                        w[nb] = __builtin_bit_cast(bf16x8_t, wv);
                    }
#pragma unroll
                    for (int mb = 0; mb < MB; mb++)
#pragma unroll
                        for (int nb = 0; nb < NB; nb++)
                            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mb], w[nb], acc[mb][nb], 0, 0, 0);
                } else {
                    f32x4 a[MB], w[NB];
#pragma unroll
                    for (int mb = 0; mb < MB; mb++) {
                        const int row = wm * WM + mb * 16 + (lane & 15) + roff;
                        a[mb] = *(const f32x4*)(lds + row * ldw + kc * 16 + (lane >> 4) * 4);
                    }
#pragma unroll
                    for (int nb = 0; nb < NB; nb++) {
                        const int nblk = (n0 + wn * WN) / 16 + nb;
                        f32x4 wv = {0.f, 0.f, 0.f, 0.f};
                        if (nblk < p.NB16) wv = ((const f32x4*)p.wp)[(wbase + nblk) * 64 + lane];
                        w[nb] = wv;
                    }
#pragma unroll
                    for (int q = 0; q < 4; q++)
#pragma unroll
                        for (int mb = 0; mb < MB; mb++)
#pragma unroll
                            for (int nb = 0; nb < NB; nb++)
                                acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb][q], w[nb][q], acc[mb][nb], 0, 0, 0);
                }
            }
        }
    }

    // Epilogue: bias, residual, branch mean, LeakyReLU, store through the ring.
#pragma unroll
    for (int mb = 0; mb < MB; mb++) {
#pragma unroll
        for (int r = 0; r < 4; r++) {
            const int t = t0 + wm * WM + mb * 16 + (lane >> 4) * 4 + r;
            if (t >= p.F) continue;
#pragma unroll
            for (int nb = 0; nb < NB; nb++) {
                const int n = n0 + wn * WN + nb * 16 + (lane & 15);
                if (n >= p.N) continue;
                float v = acc[mb][nb][r] + p.bias[n];
                int64_t fo = t;
                int co = n;
                if (p.u != 1) {
                    fo = (int64_t)t * p.u + n / p.out_C;
                    co = n % p.out_C;
                }
                const int64_t tau = tau0 * p.u + fo;
                if (p.res) v = p.res[((size_t)b * p.res_R + ring_slot(tau, p.res_R)) * p.out_C + co] + v;
                if (p.n_mean) {
                    const size_t mo = ((size_t)b * p.mean_R + ring_slot(tau, p.mean_R)) * p.out_C + co;
                    float x = p.mean[0][mo];
                    for (int i = 1; i < p.n_mean; i++) x = x + p.mean[i][mo];
                    x = x + v;
                    v = x / (float)(p.n_mean + 1);
                }
                if (p.out_act) v = lrelu(v, p.slope);
                const size_t oo = ((size_t)b * p.out_R + ring_slot(tau, p.out_R)) * p.out_C + co;
                if (p.out_elem == kF32)
                    ((float*)p.out)[oo] = v;
                else
                    ((uint16_t*)p.out)[oo] = (uint16_t)f2bf(v);
            }
        }
    }
}

// ------------------------------------------------------------- tile table

static const TileShape kTiles[] = {
    {32, 32, 2}, {32, 64, 2}, {64, 64, 2}, {64, 128, 2}, {128, 64, 4}, {128, 128, 2}, {256, 64, 4},
};

int num_tile_variants() { return (int)(sizeof(kTiles) / sizeof(kTiles[0])); }
TileShape tile_variant(int v) { return kTiles[v]; }

size_t conv_lds_bytes(int v, bool bf16, const ConvParams& p)
{
    const int rows = kTiles[v].BM + (p.k - 1) * p.d;
    const int pad = bf16 ? OpT<true>::PAD : OpT<false>::PAD;
    return (size_t)rows * (p.CB + pad) * (bf16 ? 2 : 4);
}

template <bool BF16, int BM, int BN, int WGM>
static hipError_t launch_t(const ConvParams& p, hipStream_t st)
{
    dim3 grid((unsigned)(p.B * p.tiles_t), (unsigned)((p.N + BN - 1) / BN));
    const int rows = BM + (p.k - 1) * p.d;
    const size_t lds = (size_t)rows * (p.CB + OpT<BF16>::PAD) * sizeof(typename OpT<BF16>::T);
    hipLaunchKernelGGL((conv_kernel<BF16, BM, BN, WGM>), grid, dim3(256), lds, st, p);
    return hipGetLastError();
}

template <bool BF16>
static hipError_t launch_dt(int v, const ConvParams& p, hipStream_t st)
{
    switch (v) {
    case 0: return launch_t<BF16, 32, 32, 2>(p, st);
    case 1: return launch_t<BF16, 32, 64, 2>(p, st);
    case 2: return launch_t<BF16, 64, 64, 2>(p, st);
    case 3: return launch_t<BF16, 64, 128, 2>(p, st);
    case 4: return launch_t<BF16, 128, 64, 4>(p, st);
    case 5: return launch_t<BF16, 128, 128, 2>(p, st);
    case 6: return launch_t<BF16, 256, 64, 4>(p, st);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_conv(int v, bool bf16, const ConvParams& p, hipStream_t st)
{
    return bf16 ? launch_dt<true>(v, p, st) : launch_dt<false>(v, p, st);
}

// ----------------------------------------------------------- embedding

// E[b][tau0 + f] = table[tokens[b][f / fpt]] for f in [0, n*fpt): the token
// embedding repeated to the frame clock, written through the ring.  An id
// outside [0, vocab) raises *err and writes zeros.
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* tokens, int n, int B, const void* table,
                                                    int vocab, int C, int elem, int fpt, Ring out,
                                                    const int64_t* clock, int* err)
{
    const int vpr = C / 8;
    const int64_t total = (int64_t)B * n * fpt * vpr;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int c8 = (int)(i % vpr) * 8;
    const int64_t bf = i / vpr;
    const int f = (int)(bf % (n * fpt));
    const int b = (int)(bf / (n * fpt));
    const int tok = tokens[(size_t)b * n + f / fpt];
    const int64_t slot = ring_slot(clock[0] * fpt + f, out.R);
    const size_t dst = ((size_t)b * out.R + slot) * C + c8;
    const bool ok = tok >= 0 && tok < vocab;
    if (!ok) *err = 1;
    if (elem == kF32) {
        f32x4 a = {0.f, 0.f, 0.f, 0.f}, c = a;
        if (ok) {
            const f32x4* src = (const f32x4*)((const float*)table + (size_t)tok * C + c8);
            a = src[0];
            c = src[1];
        }
        f32x4* d = (f32x4*)((float*)out.ptr + dst);
        d[0] = a;
        d[1] = c;
    } else {
        u32x4 a = {0u, 0u, 0u, 0u};
        if (ok) a = *(const u32x4*)((const uint16_t*)table + (size_t)tok * C + c8);
        *(u32x4*)((uint16_t*)out.ptr + dst) = a;
    }
}

hipError_t launch_embed(const int32_t* tokens, int n, int B, const void* table, int vocab, int C, int elem,
                        int fpt, Ring out, const int64_t* clock, int* err, hipStream_t st)
{
    const int64_t total = (int64_t)B * n * fpt * (C / 8);
    const unsigned blocks = (unsigned)((total + 255) / 256);
    hipLaunchKernelGGL(embed_kernel, dim3(blocks), dim3(256), 0, st, tokens, n, B, table, vocab, C, elem, fpt,
                       out, clock, err);
    return hipGetLastError();
}

// ------------------------------------------------ spectrum + iDFT + window

// One thread per (stream, frame m): X_kk = exp(logmag_kk) (cos ph_kk + i sin ph_kk),
// g[n] = sum_kk Tre[n][kk] Re X_kk + Tim[n][kk] Im X_kk, where the tables fold
// the real inverse DFT, the periodic Hann window and the overlap-add
// normaliser (computed in double on the host from their definitions).  The
// windowed frame g goes to the G ring, whose zeroed slots stand for frames
// before the start of the stream.
constexpr int kNFFT = 16, kBins = 9;

__global__ __launch_bounds__(256) void spectrum_kernel(const float* head, int64_t head_R, int B, int F,
                                                       const float* table, Ring g, const int64_t* clock,
                                                       int64_t fpt)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * F) return;
    const int b = (int)(i / F), m = (int)(i % F);
    const int64_t tau = clock[0] * fpt + m;
    const float* s = head + ((size_t)b * head_R + ring_slot(tau, head_R)) * (2 * kBins);
    float re[kBins], im[kBins];
#pragma unroll
    for (int kk = 0; kk < kBins; kk++) {
        const float mag = expf(s[kk]);
        float sn, cs;
        sincosf(s[kBins + kk], &sn, &cs);
        re[kk] = mag * cs;
        im[kk] = mag * sn;
    }
    float* out = (float*)g.ptr + ((size_t)b * g.R + ring_slot(tau, g.R)) * kNFFT;
#pragma unroll
    for (int n4 = 0; n4 < kNFFT; n4 += 4) {
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const float* tr = table + (n4 + e) * kBins;
            const float* ti = table + kNFFT * kBins + (n4 + e) * kBins;
            float v = 0.f;
#pragma unroll
            for (int kk = 0; kk < kBins; kk++) {
                v = fmaf(tr[kk], re[kk], v);
                v = fmaf(ti[kk], im[kk], v);
            }
            o[e] = v;
        }
        *(f32x4*)(out + n4) = o;
    }
}

hipError_t launch_spectrum(const float* head, int64_t head_R, int B, int F, const float* table, Ring g,
                           const int64_t* clock, int64_t fpt, hipStream_t st)
{
    const int64_t total = (int64_t)B * F;
    hipLaunchKernelGGL(spectrum_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, head, head_R,
                       B, F, table, g, clock, fpt);
    return hipGetLastError();
}

// ------------------------------------------------------------ overlap-add

// Sample T = hop*m0 + t: sum over the frames m = floor(T/hop) - (n_fft/hop - 1)
// .. floor(T/hop) of g_m[T - hop*m], added in ascending m from +0.
__global__ __launch_bounds__(256) void ola_kernel(Ring g, int B, int F, int hop, int n_fft, float* pcm,
                                                  const int64_t* clock, int64_t fpt)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per = (int64_t)F * hop;
    if (i >= (int64_t)B * per) return;
    const int b = (int)(i / per);
    const int64_t t = i % per;
    const int64_t m0 = clock[0] * fpt;
    const int64_t T = m0 * hop + t;
    const int64_t mu = m0 + t / hop;
    const float* base = (const float*)g.ptr + (size_t)b * g.R * kNFFT;
    float acc = 0.f;
    for (int64_t m = mu - (n_fft / hop - 1); m <= mu; m++)
        acc = acc + base[ring_slot(m, g.R) * kNFFT + (T - hop * m)];
    pcm[(size_t)b * per + t] = acc;
}

hipError_t launch_ola(Ring g, int B, int F, int hop, int n_fft, float* pcm, const int64_t* clock, int64_t fpt,
                      hipStream_t st)
{
    const int64_t total = (int64_t)B * F * hop;
    hipLaunchKernelGGL(ola_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, g, B, F, hop, n_fft,
                       pcm, clock, fpt);
    return hipGetLastError();
}

// --------------------------------------------------------------- clock

__global__ void clock_kernel(int64_t* clock, int n)
{
    if (threadIdx.x == 0) clock[0] = clock[0] + n;
}

hipError_t launch_clock(int64_t* clock, int n, hipStream_t st)
{
    hipLaunchKernelGGL(clock_kernel, dim3(1), dim3(64), 0, st, clock, n);
    return hipGetLastError();
}

}  // namespace dc
