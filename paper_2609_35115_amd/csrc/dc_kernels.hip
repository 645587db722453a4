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
#include <type_traits>

#include "dc_internal.h"
#include "dc_philox.h"


namespace dc {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

// ------------------------------------------------------------------ helpers

// float -> bfloat16 bits, round to nearest, ties to even (NaN kept quiet).
__device__ __forceinline__ uint32_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (u >> 16) | ((u & 0x007fffffu) ? 0x40u : 0u);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// Two floats -> packed bfloat16 pair (v_cvt_pk_bf16_f32: round to nearest even).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float lrelu(float v, float s) { return v >= 0.0f ? v : v * s; }

typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;

// IEEE binary16 bits -> float (exact), and two floats -> a packed binary16
// pair (round to nearest even).
__device__ __forceinline__ float h2f(uint32_t h) { return (float)__builtin_bit_cast(_Float16, (uint16_t)h); }
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi)
{
    const f16x2_t v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

// Ring element access by element type (kF32, kBF16 or kF16; a compile-time
// constant on the hot paths, so the selection folds away): four consecutive
// elements at a 4-element-aligned offset, or one.
__device__ __forceinline__ f32x4 load4(const void* base, int elem, size_t off)
{
    if (elem == kF32) return *(const f32x4*)((const float*)base + off);
    const u32x2 w = *(const u32x2*)((const uint16_t*)base + off);
    if (elem == kF16) return f32x4{h2f(w[0] & 0xffffu), h2f(w[0] >> 16), h2f(w[1] & 0xffffu), h2f(w[1] >> 16)};
    return f32x4{bf2f(w[0] & 0xffffu), bf2f(w[0] >> 16), bf2f(w[1] & 0xffffu), bf2f(w[1] >> 16)};
}

__device__ __forceinline__ float load1(const void* base, int elem, size_t off)
{
    if (elem == kF32) return ((const float*)base)[off];
    const uint32_t h = ((const uint16_t*)base)[off];
    return elem == kF16 ? h2f(h) : bf2f(h);
}

// A binary16 ring is a bf16 state's residual stream: a value it cannot hold
// (|v| >= 65520 rounds to infinity; NaN) must raise the state's error flag, so
// that the overflow poisons the state instead of silently carrying infinities
// forward.  The stores only keep, in one register per lane (`mag`, when
// given), the largest magnitude's bits (|v| as an unsigned integer orders
// finite values, infinity and NaN alike); each kernel raises the flag once,
// after its last store (raise_f16_range), so the store loops keep their shape.
constexpr uint32_t kF16Limit = 0x477ff000u;   // bits of 65520.0f

__device__ __forceinline__ uint32_t mag_bits(float v) { return __float_as_uint(v) & 0x7fffffffu; }

__device__ __forceinline__ void raise_f16_range(int* err, uint32_t mag)
{
    if (mag >= kF16Limit) atomicOr(err, kErrF16Range);
}

__device__ __forceinline__ void store4(void* base, int elem, size_t off, f32x4 v, uint32_t* mag = nullptr)
{
    if (elem == kF32) {
        *(f32x4*)((float*)base + off) = v;
    } else if (elem == kF16) {
        if (mag) *mag = max(*mag, max(max(mag_bits(v[0]), mag_bits(v[1])), max(mag_bits(v[2]), mag_bits(v[3]))));
        *(u32x2*)((uint16_t*)base + off) = u32x2{pack_f16x2(v[0], v[1]), pack_f16x2(v[2], v[3])};
    } else {
        *(u32x2*)((uint16_t*)base + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    }
}

__device__ __forceinline__ void store1(void* base, int elem, size_t off, float v, uint32_t* mag = nullptr)
{
    if (elem == kF32) {
        ((float*)base)[off] = v;
    } else if (elem == kF16) {
        if (mag) *mag = max(*mag, mag_bits(v));
        ((uint16_t*)base)[off] = __builtin_bit_cast(uint16_t, (_Float16)v);
    } else {
        ((uint16_t*)base)[off] = (uint16_t)f2bf(v);
    }
}

__device__ __forceinline__ int64_t ring_slot(int64_t tau, int64_t R)
{
    int64_t s = tau % R;
    return s < 0 ? s + R : s;
}

// ------------------------------------------------------- checked build
//
// Built with DC_DEBUG, ring accesses take their offsets from ring_at and the
// fixed-size tiles check their row ranges: an index outside its buffer sets a
// bit of dc_debug_bits (one word per lane, so the atomic has a per-lane
// address) and the access goes to element 0 of the buffer instead, so a
// checked run never leaves its buffers.  dc_debug_checks reads and clears
// the bits.  The release build computes the same offsets with no checks.
enum DebugBit : int {
    kDbgOperand = 1,      // conv: operand rows read through the input ring
    kDbgTile = 2,         // conv: operand rows of the LDS tile
    kDbgOut = 4,          // conv: output, residual, branch-mean and source rings
    kDbgPairZ = 8,        // fused pair: z ring
    kDbgPairOut = 16,     // fused pair: output and branch-mean rings
    kDbgTail = 32,        // iSTFT tail: head ring, G ring, PCM
    kDbgEmbed = 64,       // embedding: output ring
};
#ifdef DC_DEBUG
__device__ int dc_debug_bits[64];
__device__ __forceinline__ void dbg_flag(int bit) { atomicOr(&dc_debug_bits[threadIdx.x & 63], bit); }
#define DC_DBG_CHECK(cond, bit) \
    do {                        \
        if (!(cond)) dbg_flag(bit); \
    } while (0)
#else
#define DC_DBG_CHECK(cond, bit) ((void)0)
#endif

// Offset of elements c .. c + w - 1 of slot `slot` of stream b in a ring of
// B streams x R slots x C elements.
__device__ __forceinline__ size_t ring_at(int b, int B, int64_t slot, int64_t R, int c, int w, int C, int bit)
{
#ifdef DC_DEBUG
    if (b < 0 || b >= B || slot < 0 || slot >= R || c < 0 || c + w > C) {
        dbg_flag(bit);
        return 0;
    }
#endif
    return ((size_t)b * R + slot) * C + c;
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

// Load 8 channels of one frame as floats.
__device__ __forceinline__ void load8(const void* base, int elem, size_t off, float v[8])
{
    if (elem == kF32) {
        const f32x4* p = (const f32x4*)((const float*)base + off);
        f32x4 a = p[0], b = p[1];
        v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
        v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
    } else if (elem == kF16) {
        u32x4 a = *(const u32x4*)((const uint16_t*)base + off);
#pragma unroll
        for (int e = 0; e < 4; e++) {
            v[2 * e] = h2f(a[e] & 0xffffu);
            v[2 * e + 1] = h2f(a[e] >> 16);
        }
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
    for (int e = 0; e < 4; e++) w[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
    *(u32x4*)dst = w;
}

// hi = bf16(v), lo = bf16(v - hi): hi + lo carries v to about 2^-16 relative.
__device__ __forceinline__ void store8_lds_split(uint16_t* hi, uint16_t* lo, const float v[8])
{
    u32x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; e++) {
        h[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
        l[e] = pack_bf16x2(v[2 * e] - bf2f(h[e] & 0xffffu), v[2 * e + 1] - bf2f(h[e] >> 16));
    }
    *(u32x4*)hi = h;
    *(u32x4*)lo = l;
}

__device__ __forceinline__ void store8_lds(float* dst, const float v[8])
{
    f32x4 a = {v[0], v[1], v[2], v[3]}, b = {v[4], v[5], v[6], v[7]};
    *(f32x4*)dst = a;
    *(f32x4*)(dst + 4) = b;
}

// ------------------------------------------------------------ causal conv
//
// Block = 4 waves = WGM x WGN x WGK: WGM x WGN waves tile the output
// (MB x NB MFMA blocks of 16x16 each), WGK waves share one output tile and
// split K.  K runs over (channel block cb, tap j, chunk kc) in that order;
// wave wk of a K-split block takes the chunks kc = wk, wk + WGK, ... of every
// tap, accumulates them in that order in fp32, and the block adds the WGK
// partial sums in wave order: ((P_0 + P_1) + ...) + P_{WGK-1}.

// This block's output and residual rings (of its group member) and the ring
// slots of its output frame at block row 0, phase 0.
struct OutRef {
    void* out;
    const void* res;     // element type out_elem, as are the branch-mean rings
    int out_R, res_R;
    int out_s, res_s, mean_s;
    int src_s;   // ring slot of the source samples of that frame
    mutable uint32_t f16_mag = 0;   // largest binary16 store magnitude's bits (checked once, at the end)
};

// The harmonic source's contribution to output channels co .. co+3 of the
// frame whose source samples sit at ring slot `slot`:
//   sd_b[c] + sum_j sd_w[c][j] * src[j], j ascending.
__device__ __forceinline__ f32x4 src_term4(const ConvParams& p, int b, int slot, int co)
{
    const f32x4 x = *(const f32x4*)(p.src + ring_at(b, p.B, slot, p.src_R, 0, 4, 4, kDbgOut));
    f32x4 v = *(const f32x4*)(p.sd_b + co);
#pragma unroll
    for (int e = 0; e < 4; e++) {
        const f32x4 w = *(const f32x4*)(p.sd_w + (size_t)(co + e) * 4);
        float a = v[e];
#pragma unroll
        for (int j = 0; j < 4; j++) a = a + w[j] * x[j];
        v[e] = a;
    }
    return v;
}

__device__ __forceinline__ float src_term1(const ConvParams& p, int b, int slot, int co)
{
    const f32x4 x = *(const f32x4*)(p.src + ring_at(b, p.B, slot, p.src_R, 0, 4, 4, kDbgOut));
    const f32x4 w = *(const f32x4*)(p.sd_w + (size_t)co * 4);
    float a = p.sd_b[co];
#pragma unroll
    for (int j = 0; j < 4; j++) a = a + w[j] * x[j];
    return a;
}

// Slot of a frame `off` frames after a base slot, for 0 <= off < R.
__device__ __forceinline__ int slot_add(int base, int off, int R)
{
    const int s = base + off;
    return s >= R ? s - R : s;
}

__device__ __forceinline__ void store_out(const ConvParams& p, int b, const OutRef& rs, int off, int co,
                                          float v)
{
    // off: output frame offset from the block's base frame; co: output channel
    if (p.src) v = v + src_term1(p, b, slot_add(rs.src_s, off, (int)p.src_R), co);
    const int oe = p.out_elem;
    if (rs.res) v = load1(rs.res, oe, ring_at(b, p.B, slot_add(rs.res_s, off, rs.res_R), rs.res_R, co, 1, p.out_C, kDbgOut)) + v;
    if (p.n_mean) {
        const size_t mo = ring_at(b, p.B, slot_add(rs.mean_s, off, (int)p.mean_R), p.mean_R, co, 1, p.out_C, kDbgOut);
        float x = load1(p.mean[0], oe, mo);
        for (int i = 1; i < p.n_mean; i++) x = x + load1(p.mean[i], oe, mo);
        x = x + v;
        v = x / (float)(p.n_mean + 1);
    }
    if (p.out_act) v = lrelu(v, p.slope);
    store1(rs.out, oe, ring_at(b, p.B, slot_add(rs.out_s, off, rs.out_R), rs.out_R, co, 1, p.out_C, kDbgOut), v, &rs.f16_mag);
}

// Four consecutive output channels co .. co+3 of one frame (nv < 4 at the
// edge of an output whose width is not a multiple of 4).
__device__ __forceinline__ void store_out4(const ConvParams& p, int b, const OutRef& rs, int off, int co,
                                           f32x4 v, int nv)
{
    if (nv < 4 || (p.out_C & 3)) {
        for (int e = 0; e < nv; e++) store_out(p, b, rs, off, co + e, v[e]);
        return;
    }
    if (p.src) v = v + src_term4(p, b, slot_add(rs.src_s, off, (int)p.src_R), co);
    const int oe = p.out_elem;
    if (rs.res) v = load4(rs.res, oe, ring_at(b, p.B, slot_add(rs.res_s, off, rs.res_R), rs.res_R, co, 4, p.out_C, kDbgOut)) + v;
    if (p.n_mean) {
        const size_t mo = ring_at(b, p.B, slot_add(rs.mean_s, off, (int)p.mean_R), p.mean_R, co, 4, p.out_C, kDbgOut);
        f32x4 x = load4(p.mean[0], oe, mo);
        for (int i = 1; i < p.n_mean; i++) x = x + load4(p.mean[i], oe, mo);
        x = x + v;
        const float J = (float)(p.n_mean + 1);
        v = f32x4{x[0] / J, x[1] / J, x[2] / J, x[3] / J};
    }
    if (p.out_act) {
#pragma unroll
        for (int e = 0; e < 4; e++) v[e] = lrelu(v[e], p.slope);
    }
    store4(rs.out, oe, ring_at(b, p.B, slot_add(rs.out_s, off, rs.out_R), rs.out_R, co, 4, p.out_C, kDbgOut), v, &rs.f16_mag);
}

// Operand rows [t0 - halo, t0 - halo + rows) of channel block cb of stream b,
// read through the input ring (ring slot base_in holds row 0), LeakyReLU'd
// if asked, converted once to the operand type (bf16: optionally as hi + lo
// halves, the lo rows lo_off elements after the hi rows) and stored in LDS
// rows of LDW elements.  Rows at or past the call's frames are zeros.
template <bool BF16, int CB, int LDW>
__device__ __forceinline__ void stage_operand(const ConvParams& p, const void* in_ptr, int in_R, int b, int t0,
                                              int halo, int rows, int base_in, int cb,
                                              typename OpT<BF16>::T* lds, int lo_off)
{
    constexpr int VPR = CB / 8;
    for (int v = threadIdx.x; v < rows * VPR; v += 256) {
        const int r = v / VPR, c8 = (v - r * VPR) * 8;
        const int t = t0 - halo + r;
        const int ch = cb * CB + c8;
        float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (t < p.F && ch < p.in_C) {
            load8(in_ptr, p.in_elem, ring_at(b, p.B, slot_add(base_in, r, in_R), in_R, ch, 8, p.in_C, kDbgOperand), x);
            if (p.in_act) {
#pragma unroll
                for (int e = 0; e < 8; e++) x[e] = lrelu(x[e], p.slope);
            }
        }
        if constexpr (BF16) {
            if (p.split)
                store8_lds_split(lds + r * LDW + c8, lds + lo_off + r * LDW + c8, x);
            else
                store8_lds(lds + r * LDW + c8, x);
        } else {
            store8_lds(lds + r * LDW + c8, x);
        }
    }
}

// Bias of this wave's output columns: lane l holds the four consecutive
// columns 4*(l/16) .. +3 of each of its 16-column blocks (zeros past N).
template <int NB>
__device__ __forceinline__ void load_bias(const ConvParams& p, const float* bias_ptr, int n0, int colblk0, int lane,
                                          f32x4 (&bias)[NB])
{
    const int cg = (lane >> 4) * 4;
#pragma unroll
    for (int nb = 0; nb < NB; nb++) {
        const int n4 = n0 + (colblk0 + nb) * 16 + cg;
        const int nv = p.N - n4 < 4 ? p.N - n4 : 4;
#pragma unroll
        for (int e = 0; e < 4; e++) bias[nb][e] = e < nv ? bias_ptr[n4 + e] : 0.f;
    }
}

// Epilogue of a tile with one K partition: bias (preloaded by load_bias),
// residual, branch mean, LeakyReLU, stored through the output ring (rs slots
// set by the caller).  The wave holds MB x NB blocks of 16x16 whose rows start
// at tile row row0 and whose 16-column blocks start at colblk0; the weights
// are the MFMA A operand and the frames the B operand, so lane l holds output
// channels 4*(l/16) .. +3 of frame l%16 of each block: four consecutive
// channels of one frame, stored as one vector.
template <int MB, int NB, int OE>
__device__ __forceinline__ void store_tile_e(const ConvParams& p, const OutRef& rs, const f32x4 (&acc)[MB][NB],
                                             const f32x4 (&bias)[NB], int b, int t0, int n0, int row0, int colblk0,
                                             int lane)
{
    const int fl = lane & 15, cg = (lane >> 4) * 4;
    int rp[NB], co[NB], nv[NB];
#pragma unroll
    for (int nb = 0; nb < NB; nb++) {
        const int n4 = n0 + (colblk0 + nb) * 16 + cg;
        rp[nb] = p.u == 1 ? 0 : n4 / p.out_C;
        co[nb] = n4 - rp[nb] * p.out_C;
        nv[nb] = p.N - n4 < 4 ? p.N - n4 : 4;
    }
    // the wave's columns are all real and vector-aligned, and no branch mean:
    // the residual loads of row block mb + 1 are issued before row block mb
    // is finished (rows past the call's frames read its last frame and
    // store nothing).  Otherwise each output vector loads what it adds.
    const bool full = (p.out_C & 3) == 0 && n0 + (colblk0 + NB) * 16 <= p.N && p.n_mean == 0;
    if (full) {
        auto off_of = [&](int mb) {
            const int tl = row0 + mb * 16 + fl;
            return (t0 + tl < p.F ? tl : p.F - 1 - t0) * p.u;
        };
        f32x4 ld[2][NB];
        auto issue = [&](int mb, f32x4 (&q)[NB]) {
            const int off = off_of(mb);
#pragma unroll
            for (int nb = 0; nb < NB; nb++)
                q[nb] = load4(rs.res, OE, ring_at(b, p.B, slot_add(rs.res_s, off + rp[nb], rs.res_R), rs.res_R, co[nb], 4,
                                                  p.out_C, kDbgOut));
        };
        if (rs.res) issue(0, ld[0]);
#pragma unroll
        for (int mb = 0; mb < MB; mb++) {
            if (rs.res && mb + 1 < MB) issue(mb + 1, ld[(mb + 1) & 1]);
            const int off = off_of(mb);
            const bool live = t0 + row0 + mb * 16 + fl < p.F;
#pragma unroll
            for (int nb = 0; nb < NB; nb++) {
                f32x4 v = acc[mb][nb] + bias[nb];
                if (p.src) v = v + src_term4(p, b, slot_add(rs.src_s, off + rp[nb], (int)p.src_R), co[nb]);
                if (rs.res) v = ld[mb & 1][nb] + v;
                if (p.out_act) {
#pragma unroll
                    for (int e = 0; e < 4; e++) v[e] = lrelu(v[e], p.slope);
                }
                if (!live) continue;
                store4(rs.out, OE, ring_at(b, p.B, slot_add(rs.out_s, off + rp[nb], rs.out_R), rs.out_R, co[nb], 4, p.out_C,
                                           kDbgOut), v, &rs.f16_mag);
            }
        }
    } else {
#pragma unroll
        for (int mb = 0; mb < MB; mb++) {
            const int tl = row0 + mb * 16 + fl;
            if (t0 + tl >= p.F) continue;
#pragma unroll
            for (int nb = 0; nb < NB; nb++) {
                if (nv[nb] <= 0) continue;
                f32x4 v = acc[mb][nb];
                store_out4(p, b, rs, tl * p.u + rp[nb], co[nb], v + bias[nb], nv[nb]);
            }
        }
    }
}

// store_tile_e for the output's element type (fp32 operands write fp32 only).
template <bool BF16, int MB, int NB>
__device__ __forceinline__ void store_tile(const ConvParams& p, const OutRef& rs, const f32x4 (&acc)[MB][NB],
                                           const f32x4 (&bias)[NB], int b, int t0, int n0, int row0, int colblk0,
                                           int lane)
{
    if (!BF16 || p.out_elem == kF32)
        store_tile_e<MB, NB, kF32>(p, rs, acc, bias, b, t0, n0, row0, colblk0, lane);
    else if (p.out_elem == kF16)
        store_tile_e<MB, NB, kF16>(p, rs, acc, bias, b, t0, n0, row0, colblk0, lane);
    else
        store_tile_e<MB, NB, kBF16>(p, rs, acc, bias, b, t0, n0, row0, colblk0, lane);
}

template <bool BF16, int MB, int NB, int WGM, int WGN, int WGK, int KCH>
__global__ __launch_bounds__(256) void conv_kernel(const ConvGroup g)
{
    // shared fields from member 0; this block's member supplies the rest
    const ConvParams& p = g.p;
    const void* in_ptr = p.in;
    int in_R = (int)p.in_R;
    const void* w_ptr = p.wp;
    const float* bias_ptr = p.bias;
    OutRef rs{p.out, p.res, (int)p.out_R, (int)p.res_R, 0, 0, 0};
    int k = p.k;
    if (blockIdx.z > 0) {
        const ConvMember& m = g.m[blockIdx.z - 1];
        in_ptr = m.in;
        in_R = (int)m.in_R;
        w_ptr = m.wp;
        bias_ptr = m.bias;
        rs.out = m.out;
        rs.out_R = (int)m.out_R;
        rs.res = m.res;
        rs.res_R = (int)m.res_R;
        k = m.k;
    }
    using Tr = OpT<BF16>;
    using T = typename Tr::T;
    using Frag = typename std::conditional<BF16, u32x4, f32x4>::type;
    constexpr int BM = 16 * MB * WGM, BN = 16 * NB * WGN, S = WGK;
    constexpr int CB = Tr::KQ * KCH;        // channels per block
    constexpr int KPW = KCH / WGK;          // this wave's K chunks per tap
    constexpr int LDW = CB + Tr::PAD;       // LDS row stride (elements)
    constexpr int VPR = CB / 8;             // 8-channel vectors per LDS row
    static_assert(WGM * WGN * WGK == 4 && KCH % WGK == 0, "tile shape");

    extern __shared__ __align__(16) unsigned char smem[];
    T* lds = reinterpret_cast<T*>(smem);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar index math
    const int wk = wave % WGK, wm = (wave / WGK) % WGM, wn = wave / (WGK * WGM);
    const int b = blockIdx.x / p.tiles_t;
    const int t0 = (blockIdx.x - b * p.tiles_t) * BM;
    const int n0 = blockIdx.y * BN;
    const int halo = (k - 1) * p.d;
    const int rows = BM + halo;
    const int64_t tau0 = p.clock[0] * p.in_fpt;
    const int base_in = (int)ring_slot(tau0 + t0 - halo, in_R);
    const int nblk0 = n0 / 16 + wn * NB;
    const Frag* wp = reinterpret_cast<const Frag*>(w_ptr);

    // K-split tiles hold at most one output vector per thread in the
    // epilogue: its bias and residual are loaded here, before the K loop, so
    // the epilogue does not wait for them (a vector with a branch mean, or at
    // the edge of the output, loads what it adds there instead)
    const int e_idx = tid * 4;
    const int e_tl = e_idx / BN, e_n4 = n0 + (e_idx - (e_idx / BN) * BN);
    const bool e_live = WGK > 1 && e_idx < BM * BN && t0 + e_tl < p.F && e_n4 < p.N;
    // Both are kept as loaded (the residual as raw bits, converted in the
    // epilogue, and bias elements past the layer's columns as whatever the
    // clamped load returned, never stored), so that nothing reads these
    // registers before the epilogue and the loads stay in flight through the
    // operand staging instead of being waited for ahead of it.
    f32x4 e_bias = {0.f, 0.f, 0.f, 0.f};
    u32x4 e_raw = {0u, 0u, 0u, 0u};
    bool e_pre = false;
    if constexpr (WGK > 1) {
        static_assert(BM * BN <= 4 * 256, "one output vector per thread");
        if (e_live) {
            const int nv = p.N - e_n4 < 4 ? p.N - e_n4 : 4;
#pragma unroll
            for (int e = 0; e < 4; e++) e_bias[e] = bias_ptr[e_n4 + (e < nv ? e : 0)];
            e_pre = nv == 4 && (p.out_C & 3) == 0 && p.n_mean == 0;
            if (e_pre && rs.res) {
                const int rpn = p.u == 1 ? 0 : e_n4 / p.out_C;
                const int res_s = (int)ring_slot((tau0 + t0) * p.u, rs.res_R);
                const size_t ro = ring_at(b, p.B, slot_add(res_s, e_tl * p.u + rpn, rs.res_R), rs.res_R,
                                          e_n4 - rpn * p.out_C, 4, p.out_C, kDbgOut);
                if (p.out_elem == kF32) {
                    e_raw = *(const u32x4*)((const float*)rs.res + ro);
                } else {
                    const u32x2 h = *(const u32x2*)((const uint16_t*)rs.res + ro);
                    e_raw[0] = h[0];
                    e_raw[1] = h[1];
                }
            }
        }
    }

    f32x4 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; i++)
#pragma unroll
        for (int j = 0; j < NB; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Weight fragments of this wave for tap j of channel block cb.  Column
    // blocks past the layer's last one re-read that block (unconditional
    // loads keep the compiler's wait counts exact); their columns are never
    // stored.
    int nblk[NB];
#pragma unroll
    for (int nb = 0; nb < NB; nb++) nblk[nb] = nblk0 + nb < p.NB16 ? nblk0 + nb : p.NB16 - 1;
    // K steps of one channel block: step s = tap j * KPW + this wave's chunk
    // ki of the tap.  Weight fragments run two steps ahead and frame
    // fragments one step ahead, each in a ring of three register buffers,
    // so neither the L2 nor the LDS latency sits between two steps' MFMAs.
    // Every accumulator still adds its steps in ascending (tap, chunk) order.
    using AFrag = typename std::conditional<BF16, u32x4, f32x4>::type;   // frames of one K chunk
    constexpr int VEC = BF16 ? 8 : 4;       // operand elements per lane per K chunk
    const T* a_lane = lds + (wm * 16 * MB + (lane & 15)) * LDW + (lane >> 4) * VEC + wk * Tr::KQ;
    const int lo_off = rows * LDW;          // low halves of a split operand
    const int nsteps = k * KPW;
    auto load_w = [&](int cb, int st, Frag (&w)[NB]) {
        st = st < nsteps ? st : nsteps - 1;
        const int j = st / KPW, ki = st - (st / KPW) * KPW;
        const Frag* wt = wp + ((size_t)(cb * k + j) * KCH + ki * WGK + wk) * p.NB16 * 64 + lane;
#pragma unroll
        for (int nb = 0; nb < NB; nb++) w[nb] = wt[(size_t)nblk[nb] * 64];
    };
    auto step_a = [&](int st) {   // this lane's frame fragment of step st, block row 0
        const int j = st / KPW, ki = st - (st / KPW) * KPW;
        DC_DBG_CHECK(wm * 16 * MB + 16 * MB - 1 + j * p.d < rows, kDbgTile);
        return a_lane + j * p.d * LDW + ki * WGK * Tr::KQ;
    };
    auto load_a = [&](int st, AFrag (&a)[MB]) {
        const T* as = step_a(st < nsteps ? st : nsteps - 1);
#pragma unroll
        for (int mb = 0; mb < MB; mb++) a[mb] = *(const AFrag*)(as + mb * 16 * LDW);
    };
    auto mma = [&](int st, const Frag (&w)[NB], const AFrag (&a)[MB]) {
        if constexpr (BF16) {
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[nb]),
                                                                         __builtin_bit_cast(bf16x8_t, a[mb]),
                                                                         acc[mb][nb], 0, 0, 0);
            if (p.split) {   // the low halves, right after the high halves of the same step
                const T* as = step_a(st) + lo_off;
                bf16x8_t lo[MB];
#pragma unroll
                for (int mb = 0; mb < MB; mb++) lo[mb] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(as + mb * 16 * LDW));
#pragma unroll
                for (int mb = 0; mb < MB; mb++)
#pragma unroll
                    for (int nb = 0; nb < NB; nb++)
                        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[nb]),
                                                                             lo[mb], acc[mb][nb], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; q++)
#pragma unroll
                for (int mb = 0; mb < MB; mb++)
#pragma unroll
                    for (int nb = 0; nb < NB; nb++)
                        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[nb][q], a[mb][q], acc[mb][nb], 0, 0, 0);
        }
    };

    // Operand rows [t0 - halo, t0 + BM) of channel block cb, through the ring.
    auto load_operand = [&](int cb) {
        stage_operand<BF16, CB, LDW>(p, in_ptr, in_R, b, t0, halo, rows, base_in, cb, lds, lo_off);
    };

    // Large per-wave tiles (at least 8 fragments): the step pipeline below.
    // Small ones: whole taps in pairs (two tap buffers of weights, frames read
    // as needed), where the per-step bookkeeping would outweigh the MFMAs.
    constexpr bool PIPE = MB * NB >= 8;
    if constexpr (!PIPE) {
        // weight fragments of this wave for tap j of channel block cb
        auto load_tap = [&](int cb, int j, Frag (&w)[KPW][NB]) {
            const Frag* wt = wp + (size_t)(cb * k + j) * KCH * p.NB16 * 64 + lane;
#pragma unroll
            for (int ki = 0; ki < KPW; ki++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++) w[ki][nb] = wt[((size_t)(ki * WGK + wk) * p.NB16 + nblk[nb]) * 64];
        };
        // MFMAs of tap j: this lane's fragment address is fixed; a tap adds a
        // row offset, a block / chunk an immediate
        auto compute_tap = [&](int j, const Frag (&w)[KPW][NB]) {
            DC_DBG_CHECK(wm * 16 * MB + 16 * MB - 1 + j * p.d < rows, kDbgTile);
            const T* aj = a_lane + j * p.d * LDW;
#pragma unroll
            for (int ki = 0; ki < KPW; ki++) {
                const int koff = ki * WGK * Tr::KQ;
                AFrag a[MB];
#pragma unroll
                for (int mb = 0; mb < MB; mb++) a[mb] = *(const AFrag*)(aj + mb * 16 * LDW + koff);
                if constexpr (BF16) {
#pragma unroll
                    for (int mb = 0; mb < MB; mb++)
#pragma unroll
                        for (int nb = 0; nb < NB; nb++)
                            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8_t, w[ki][nb]), __builtin_bit_cast(bf16x8_t, a[mb]),
                                acc[mb][nb], 0, 0, 0);
                    if (p.split) {   // the low halves, right after the high halves of the same step
#pragma unroll
                        for (int mb = 0; mb < MB; mb++) a[mb] = *(const AFrag*)(aj + lo_off + mb * 16 * LDW + koff);
#pragma unroll
                        for (int mb = 0; mb < MB; mb++)
#pragma unroll
                            for (int nb = 0; nb < NB; nb++)
                                acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    __builtin_bit_cast(bf16x8_t, w[ki][nb]), __builtin_bit_cast(bf16x8_t, a[mb]),
                                    acc[mb][nb], 0, 0, 0);
                    }
                } else {
#pragma unroll
                    for (int q = 0; q < 4; q++)
#pragma unroll
                        for (int mb = 0; mb < MB; mb++)
#pragma unroll
                            for (int nb = 0; nb < NB; nb++)
                                acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[ki][nb][q], a[mb][q], acc[mb][nb],
                                                                                  0, 0, 0);
                }
            }
        };
        Frag w0[KPW][NB], w1[KPW][NB];
        for (int cb = 0; cb < p.n_cb; cb++) {
            __syncthreads();
            load_tap(cb, 0, w0);
            load_operand(cb);
            __syncthreads();
            int j = 0;
            // scheduling barriers keep each tap's loads ahead of the previous
            // tap's MFMAs (the scheduler would otherwise sink them to their use)
            for (; j + 1 < k; j += 2) {
                load_tap(cb, j + 1, w1);
                __builtin_amdgcn_sched_barrier(0);
                compute_tap(j, w0);
                __builtin_amdgcn_sched_barrier(0);
                load_tap(cb, j + 2 < k ? j + 2 : j + 1, w0);
                __builtin_amdgcn_sched_barrier(0);
                compute_tap(j + 1, w1);
                __builtin_amdgcn_sched_barrier(0);
            }
            if (j < k) compute_tap(j, w0);
        }
    } else {
    Frag W0[NB], W1[NB], W2[NB];
    AFrag A0[MB], A1[MB], A2[MB];
    for (int cb = 0; cb < p.n_cb; cb++) {
        __syncthreads();
        load_w(cb, 0, W0);
        load_w(cb, 1, W1);
        load_operand(cb);
        __syncthreads();
        load_a(0, A0);
        // three steps per iteration: step s uses W[s % 3] and A[s % 3]
        for (int st = 0; st < nsteps; st += 3) {
            load_w(cb, st + 2, W2);
            load_a(st + 1, A1);
            __builtin_amdgcn_sched_barrier(0);
            mma(st, W0, A0);
            __builtin_amdgcn_sched_barrier(0);
            if (st + 1 >= nsteps) break;
            load_w(cb, st + 3, W0);
            load_a(st + 2, A2);
            __builtin_amdgcn_sched_barrier(0);
            mma(st + 1, W1, A1);
            __builtin_amdgcn_sched_barrier(0);
            if (st + 2 >= nsteps) break;
            load_w(cb, st + 4, W1);
            load_a(st + 3, A0);
            __builtin_amdgcn_sched_barrier(0);
            mma(st + 2, W2, A2);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    }

    // ---- epilogue: bias, residual, branch mean, LeakyReLU, store through the rings
    const int64_t tau_out0 = (tau0 + t0) * p.u;   // output frame of block row 0, phase 0
    rs.out_s = (int)ring_slot(tau_out0, rs.out_R);
    rs.res_s = rs.res ? (int)ring_slot(tau_out0, rs.res_R) : 0;
    rs.mean_s = p.n_mean ? (int)ring_slot(tau_out0, p.mean_R) : 0;
    rs.src_s = p.src ? (int)ring_slot(tau_out0, p.src_R) : 0;

    // The weights are the MFMA A operand and the frames the B operand, so lane
    // l holds output channels 4*(l/16) .. +3 of frame l%16 of each 16x16 block:
    // four consecutive channels of one frame, stored as one vector.
    const int fl = lane & 15, cg = (lane >> 4) * 4;
    if constexpr (WGK == 1) {
        f32x4 bias[NB];
        load_bias<NB>(p, bias_ptr, n0, wn * NB, lane, bias);
        store_tile<BF16, MB, NB>(p, rs, acc, bias, b, t0, n0, wm * 16 * MB, wn * NB, lane);
    } else {
        // partial sums of every partition through LDS, added in partition order
        __syncthreads();
        float* red = reinterpret_cast<float*>(smem);
#pragma unroll
        for (int mb = 0; mb < MB; mb++)
#pragma unroll
            for (int nb = 0; nb < NB; nb++) {
                const int row = wm * 16 * MB + mb * 16 + fl;
                const int col = (wn * NB + nb) * 16 + cg;
                *(f32x4*)(red + (wk * BM + row) * BN + col) = acc[mb][nb];
            }
        __syncthreads();
        if (e_live) {
            f32x4 v = *(const f32x4*)(red + e_idx);
#pragma unroll
            for (int q = 1; q < S; q++) v = v + *(const f32x4*)(red + q * BM * BN + e_idx);
            v = v + e_bias;
            const int rpn = p.u == 1 ? 0 : e_n4 / p.out_C;
            const int off = e_tl * p.u + rpn, co = e_n4 - rpn * p.out_C;
            if (e_pre) {   // the vector path of store_out4, with the residual loaded up front
                if (p.src) v = v + src_term4(p, b, slot_add(rs.src_s, off, (int)p.src_R), co);
                if (rs.res) {
                    const f32x4 e_res =
                        p.out_elem == kF32 ? __builtin_bit_cast(f32x4, e_raw)
                        : p.out_elem == kF16
                            ? f32x4{h2f(e_raw[0] & 0xffffu), h2f(e_raw[0] >> 16), h2f(e_raw[1] & 0xffffu), h2f(e_raw[1] >> 16)}
                            : f32x4{bf2f(e_raw[0] & 0xffffu), bf2f(e_raw[0] >> 16), bf2f(e_raw[1] & 0xffffu),
                                    bf2f(e_raw[1] >> 16)};
                    v = e_res + v;
                }
                if (p.out_act) {
#pragma unroll
                    for (int e = 0; e < 4; e++) v[e] = lrelu(v[e], p.slope);
                }
                store4(rs.out, p.out_elem, ring_at(b, p.B, slot_add(rs.out_s, off, rs.out_R), rs.out_R, co, 4, p.out_C, kDbgOut),
                       v, &rs.f16_mag);
            } else {
                store_out4(p, b, rs, off, co, v, p.N - e_n4 < 4 ? p.N - e_n4 : 4);
            }
        }
    }
    raise_f16_range(p.err, rs.f16_mag);
}

// ------------------------------------------- conv with an LDS weight ring
//
// bf16 operands, one K partition.  The same tiling and K order as
// conv_kernel (so the same bits for the same channel block), but the weight
// fragments of each K step go through a ring of kRing LDS slots that every
// wave of the block reads: the block fetches each fragment once (not once per
// wave row), with direct global->LDS loads that hold no registers while in
// flight, kRing - 2 steps ahead.  Each step is published by one barrier; a
// wave reads the fragments of step s + 1 (weights from the ring, frames from
// the operand tile) while its MFMAs of step s run.
constexpr int kRing = 4;

#define DC_LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

template <int MB, int NB, int WGM, int WGN, int KCH>
__global__ __launch_bounds__(256, 2) void wconv_kernel(const ConvGroup g)
{
    const ConvParams& p = g.p;
    const void* in_ptr = p.in;
    int in_R = (int)p.in_R;
    const void* w_ptr = p.wp;
    const float* bias_ptr = p.bias;
    OutRef rs{p.out, p.res, (int)p.out_R, (int)p.res_R, 0, 0, 0};
    int k = p.k;
    if (blockIdx.z > 0) {
        const ConvMember& m = g.m[blockIdx.z - 1];
        in_ptr = m.in;
        in_R = (int)m.in_R;
        w_ptr = m.wp;
        bias_ptr = m.bias;
        rs.out = m.out;
        rs.out_R = (int)m.out_R;
        rs.res = m.res;
        rs.res_R = (int)m.res_R;
        k = m.k;
    }
    using T = uint16_t;
    constexpr int BM = 16 * MB * WGM, BN = 16 * NB * WGN;
    constexpr int CB = 32 * KCH, LDW = CB + OpT<true>::PAD;
    constexpr int NFR = BN / 16;            // weight fragments (16 columns x 32 channels) per K step
    constexpr int FPW = NFR / 4;            // of which each wave loads FPW
    static_assert(WGM * WGN == 4 && NFR % 4 == 0, "wide tile shape");

    extern __shared__ __align__(16) unsigned char smem[];
    u32x4* ring = reinterpret_cast<u32x4*>(smem);                            // [kRing][NFR][64 lanes]
    T* lds = reinterpret_cast<T*>(smem + kRing * NFR * 1024);                // operand rows

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WGM, wn = wave / WGM;
    const int b = blockIdx.x / p.tiles_t;
    const int t0 = (blockIdx.x - b * p.tiles_t) * BM;
    const int n0 = blockIdx.y * BN;
    const int halo = (k - 1) * p.d;
    const int rows = BM + halo;
    const int64_t tau0 = p.clock[0] * p.in_fpt;
    const int base_in = (int)ring_slot(tau0 + t0 - halo, in_R);
    const int lo_off = rows * LDW;
    const int kk = k * KCH;                 // K steps per channel block
    const int nsteps = p.n_cb * kk;
    const u32x4* wp = reinterpret_cast<const u32x4*>(w_ptr);

    // direct loads of K step st into ring slot st % kRing (steps past the
    // last load the last step again, into a slot already consumed, so every
    // wave issues the same number of loads per step and its wait counts stay
    // exact); column blocks past the layer's last re-read it
    int fcol[FPW];
#pragma unroll
    for (int q = 0; q < FPW; q++) {
        const int c = n0 / 16 + wave + 4 * q;
        fcol[q] = c < p.NB16 ? c : p.NB16 - 1;
    }
    auto issue = [&](int st) {
        u32x4* dst = ring + (st % kRing) * NFR * 64;
        st = st < nsteps ? st : nsteps - 1;
        const u32x4* src = wp + (size_t)st * p.NB16 * 64 + lane;
#pragma unroll
        for (int q = 0; q < FPW; q++)
            __builtin_amdgcn_global_load_lds((const void*)(src + (size_t)fcol[q] * 64),
                                             DC_LDS_PTR(dst + (wave + 4 * q) * 64), 16, 0, 0);
    };

    f32x4 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; i++)
#pragma unroll
        for (int j = 0; j < NB; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const T* a_lane = lds + (wm * 16 * MB + (lane & 15)) * LDW + (lane >> 4) * 8;
    // fragments of K step st (local step sl within its channel block)
    auto readf = [&](int st, int sl, u32x4 (&a)[MB], u32x4 (&w)[NB]) {
        const int j = sl / KCH, kc = sl - (sl / KCH) * KCH;
        DC_DBG_CHECK(wm * 16 * MB + 16 * MB - 1 + j * p.d < rows, kDbgTile);
        const u32x4* wr = ring + (st % kRing) * NFR * 64 + wn * NB * 64 + lane;
#pragma unroll
        for (int nb = 0; nb < NB; nb++) w[nb] = wr[nb * 64];
        const T* as = a_lane + j * p.d * LDW + kc * 32;
#pragma unroll
        for (int mb = 0; mb < MB; mb++) a[mb] = *(const u32x4*)(as + mb * 16 * LDW);
    };
    auto mma = [&](int sl, const u32x4 (&a)[MB], const u32x4 (&w)[NB]) {
#pragma unroll
        for (int mb = 0; mb < MB; mb++)
#pragma unroll
            for (int nb = 0; nb < NB; nb++)
                acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[nb]),
                                                                     __builtin_bit_cast(bf16x8_t, a[mb]),
                                                                     acc[mb][nb], 0, 0, 0);
        if (p.split) {   // the low halves, right after the high halves of the same step
            const int j = sl / KCH, kc = sl - (sl / KCH) * KCH;
            const T* as = a_lane + lo_off + j * p.d * LDW + kc * 32;
            bf16x8_t lo[MB];
#pragma unroll
            for (int mb = 0; mb < MB; mb++) lo[mb] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(as + mb * 16 * LDW));
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[nb]), lo[mb],
                                                                         acc[mb][nb], 0, 0, 0);
        }
    };
    // own loads of the next step done (kRing - 3 later steps may stay in
    // flight), then the barrier publishes everyone's
    auto wait_step = [&] {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((kRing - 3) * FPW));
        __builtin_amdgcn_s_barrier();
    };

    for (int q = 0; q < kRing - 1; q++) issue(q);
    f32x4 bias[NB];   // loaded now, used by the epilogue
    load_bias<NB>(p, bias_ptr, n0, wn * NB, lane, bias);
    u32x4 a0[MB], w0[NB], a1[MB], w1[NB];
    for (int cb = 0; cb < p.n_cb; cb++) {
        const int s0 = cb * kk;
        if (cb > 0) __syncthreads();   // every wave is done with the previous channel block's rows
        stage_operand<true, CB, LDW>(p, in_ptr, in_R, b, t0, halo, rows, base_in, cb, lds, lo_off);
        // the rows (and, since their loads wait for every earlier load, the
        // ring slots of steps up to s0 + kRing - 2) are in place
        __syncthreads();
        readf(s0, 0, a0, w0);
        int sl = 0;
        for (; sl + 1 < kk; sl += 2) {
            wait_step();
            issue(s0 + sl + kRing - 1);
            readf(s0 + sl + 1, sl + 1, a1, w1);
            __builtin_amdgcn_sched_barrier(0);
            mma(sl, a0, w0);
            __builtin_amdgcn_sched_barrier(0);
            wait_step();
            issue(s0 + sl + kRing);
            const int nx = sl + 2 < kk ? sl + 2 : sl + 1;   // (the block's last step re-reads itself)
            readf(s0 + nx, nx, a0, w0);
            __builtin_amdgcn_sched_barrier(0);
            mma(sl + 1, a1, w1);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (sl < kk) mma(sl, a0, w0);
    }

    const int64_t tau_out0 = (tau0 + t0) * p.u;
    rs.out_s = (int)ring_slot(tau_out0, rs.out_R);
    rs.res_s = rs.res ? (int)ring_slot(tau_out0, rs.res_R) : 0;
    rs.mean_s = p.n_mean ? (int)ring_slot(tau_out0, p.mean_R) : 0;
    rs.src_s = p.src ? (int)ring_slot(tau_out0, p.src_R) : 0;
    store_tile<true, MB, NB>(p, rs, acc, bias, b, t0, n0, wm * 16 * MB, wn * NB, lane);
    raise_f16_range(p.err, rs.f16_mag);
}

// ------------------------------------------------- dynamic LDS over 64 KB
//
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

// ------------------------------------------------------------- tile table

// Every shape exists for both operand types; KCH is the channel block in
// MFMA K chunks (bf16: 32 channels, fp32: 16 channels per chunk).
static const TileShape kTiles[] = {
    // MB NB WGM WGN WGK KCH
    {1, 1, 1, 1, 4, 4},    // 0: 16x16, K in 4 partitions across waves
    {1, 1, 1, 1, 4, 8},    // 1
    {1, 1, 1, 1, 4, 16},   // 2
    {1, 2, 1, 1, 4, 4},    // 3: 16x32, 4 partitions
    {1, 2, 1, 1, 4, 8},    // 4
    {2, 2, 1, 1, 4, 4},    // 5: 32x32, 4 partitions
    {1, 1, 2, 2, 1, 2},    // 6: 32x32
    {1, 1, 2, 2, 1, 4},    // 7
    {1, 2, 2, 2, 1, 4},    // 8: 32x64
    {2, 2, 2, 2, 1, 2},    // 9: 64x64
    {2, 2, 2, 2, 1, 4},    // 10
    {2, 4, 2, 2, 1, 4},    // 11: 64x128
    {2, 4, 4, 1, 1, 2},    // 12: 128x64
    {2, 4, 4, 1, 1, 4},    // 13
    {4, 4, 2, 2, 1, 4},    // 14: 128x128
    {4, 4, 4, 1, 1, 2},    // 15: 256x64
    {4, 4, 4, 1, 1, 4},    // 16
    {1, 1, 1, 1, 4, 32},   // 17: 16x16, 4 partitions, wide channel block
    {1, 2, 1, 1, 4, 16},   // 18: 16x32
    {1, 1, 2, 2, 1, 1},    // 19: 32x32, narrow channel block
    // weights through the LDS ring (wconv_kernel; bf16 only)
    {4, 4, 2, 2, 1, 4, 1}, // 20: 128x128
    {2, 4, 2, 2, 1, 4, 1}, // 21: 64x128
    {4, 4, 4, 1, 1, 2, 1}, // 22: 256x64, 64-channel blocks
    {2, 4, 4, 1, 1, 2, 1}, // 23: 128x64, 64-channel blocks
    {4, 4, 4, 1, 1, 4, 1}, // 24: 256x64
    {2, 4, 4, 1, 1, 4, 1}, // 25: 128x64
    {1, 4, 4, 1, 1, 4, 1}, // 26: 64x64
    {2, 2, 1, 1, 4, 8},    // 27: 32x32, 4 partitions, 8-chunk channel block
    {2, 2, 4, 1, 1, 2},    // 28: 128x32, for outputs of at most 32 columns
};

int num_tile_variants() { return (int)(sizeof(kTiles) / sizeof(kTiles[0])); }
TileShape tile_variant(int v) { return kTiles[v]; }

size_t conv_lds_bytes(int v, bool bf16, const ConvParams& p)
{
    const TileShape& t = kTiles[v];
    const int rows = t.BM() + (p.k - 1) * p.d;
    const int pad = bf16 ? OpT<true>::PAD : OpT<false>::PAD;
    const int cb = t.KCH * (bf16 ? OpT<true>::KQ : OpT<false>::KQ);
    const size_t a = (size_t)rows * (cb + pad) * (bf16 ? 2 : 4) * (bf16 && p.split ? 2 : 1);
    if (t.W) return (size_t)kRing * (t.BN() / 16) * 1024 + a;
    const size_t red = t.WGK > 1 ? (size_t)t.S() * t.BM() * t.BN() * 4 : 0;
    return a > red ? a : red;
}

template <bool BF16, int MB, int NB, int WGM, int WGN, int WGK, int KCH>
static hipError_t launch_t(const ConvGroup& g, int count, size_t lds, hipStream_t st)
{
    constexpr int BN = 16 * NB * WGN;
    const ConvParams& p = g.p;   // members share B, F, N and the tiling
    dim3 grid((unsigned)(p.B * p.tiles_t), (unsigned)((p.N + BN - 1) / BN), (unsigned)count);
    static size_t lds_set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&conv_kernel<BF16, MB, NB, WGM, WGN, WGK, KCH>), lds,
                                   lds_set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((conv_kernel<BF16, MB, NB, WGM, WGN, WGK, KCH>), grid, dim3(256), lds, st, g);
    return hipGetLastError();
}

template <int MB, int NB, int WGM, int WGN, int KCH>
static hipError_t launch_w(const ConvGroup& g, int count, size_t lds, hipStream_t st)
{
    constexpr int BN = 16 * NB * WGN;
    const ConvParams& p = g.p;
    dim3 grid((unsigned)(p.B * p.tiles_t), (unsigned)((p.N + BN - 1) / BN), (unsigned)count);
    static size_t lds_set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&wconv_kernel<MB, NB, WGM, WGN, KCH>), lds, lds_set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wconv_kernel<MB, NB, WGM, WGN, KCH>), grid, dim3(256), lds, st, g);
    return hipGetLastError();
}

template <bool BF16>
static hipError_t launch_dt(int v, const ConvGroup& p, int count, size_t lds, hipStream_t st)
{
    if (v >= 20 && v <= 26) {
        if (!BF16) return hipErrorInvalidValue;
        switch (v) {
        case 20: return launch_w<4, 4, 2, 2, 4>(p, count, lds, st);
        case 21: return launch_w<2, 4, 2, 2, 4>(p, count, lds, st);
        case 22: return launch_w<4, 4, 4, 1, 2>(p, count, lds, st);
        case 23: return launch_w<2, 4, 4, 1, 2>(p, count, lds, st);
        case 24: return launch_w<4, 4, 4, 1, 4>(p, count, lds, st);
        case 25: return launch_w<2, 4, 4, 1, 4>(p, count, lds, st);
        case 26: return launch_w<1, 4, 4, 1, 4>(p, count, lds, st);
        default: return hipErrorInvalidValue;
        }
    }
    switch (v) {
    case 0: return launch_t<BF16, 1, 1, 1, 1, 4, 4>(p, count, lds, st);
    case 1: return launch_t<BF16, 1, 1, 1, 1, 4, 8>(p, count, lds, st);
    case 2: return launch_t<BF16, 1, 1, 1, 1, 4, 16>(p, count, lds, st);
    case 3: return launch_t<BF16, 1, 2, 1, 1, 4, 4>(p, count, lds, st);
    case 4: return launch_t<BF16, 1, 2, 1, 1, 4, 8>(p, count, lds, st);
    case 5: return launch_t<BF16, 2, 2, 1, 1, 4, 4>(p, count, lds, st);
    case 6: return launch_t<BF16, 1, 1, 2, 2, 1, 2>(p, count, lds, st);
    case 7: return launch_t<BF16, 1, 1, 2, 2, 1, 4>(p, count, lds, st);
    case 8: return launch_t<BF16, 1, 2, 2, 2, 1, 4>(p, count, lds, st);
    case 9: return launch_t<BF16, 2, 2, 2, 2, 1, 2>(p, count, lds, st);
    case 10: return launch_t<BF16, 2, 2, 2, 2, 1, 4>(p, count, lds, st);
    case 11: return launch_t<BF16, 2, 4, 2, 2, 1, 4>(p, count, lds, st);
    case 12: return launch_t<BF16, 2, 4, 4, 1, 1, 2>(p, count, lds, st);
    case 13: return launch_t<BF16, 2, 4, 4, 1, 1, 4>(p, count, lds, st);
    case 14: return launch_t<BF16, 4, 4, 2, 2, 1, 4>(p, count, lds, st);
    case 15: return launch_t<BF16, 4, 4, 4, 1, 1, 2>(p, count, lds, st);
    case 16: return launch_t<BF16, 4, 4, 4, 1, 1, 4>(p, count, lds, st);
    case 17: return launch_t<BF16, 1, 1, 1, 1, 4, 32>(p, count, lds, st);
    case 18: return launch_t<BF16, 1, 2, 1, 1, 4, 16>(p, count, lds, st);
    case 19: return launch_t<BF16, 1, 1, 2, 2, 1, 1>(p, count, lds, st);
    case 27: return launch_t<BF16, 2, 2, 1, 1, 4, 8>(p, count, lds, st);
    case 28: return launch_t<BF16, 2, 2, 4, 1, 1, 2>(p, count, lds, st);
    default: return hipErrorInvalidValue;
    }
}

// Members beyond the first may differ from it only in the ConvMember fields.
static bool same_shape(const ConvParams& a, const ConvParams& b)
{
    return a.in_C == b.in_C && a.in_elem == b.in_elem &&
           a.in_act == b.in_act && a.split == b.split && a.CB == b.CB && a.n_cb == b.n_cb && a.d == b.d &&
           a.N == b.N && a.NB16 == b.NB16 && a.out_C == b.out_C && a.out_elem == b.out_elem &&
           a.out_act == b.out_act && a.u == b.u && a.n_mean == b.n_mean && a.B == b.B && a.F == b.F &&
           a.tiles_t == b.tiles_t && a.clock == b.clock && a.in_fpt == b.in_fpt && a.slope == b.slope &&
           (a.res == nullptr) == (b.res == nullptr) && a.src == b.src && (a.n_mean == 0 || (a.mean_R == b.mean_R &&
           a.mean[0] == b.mean[0] && a.mean[1] == b.mean[1] && a.mean[2] == b.mean[2]));
}

hipError_t launch_conv(int v, bool bf16, const ConvParams* ps, int count, hipStream_t st)
{
    if (count < 1 || count > kMaxGroup) return hipErrorInvalidValue;
    ConvGroup g{};
    g.p = ps[0];
    size_t lds = conv_lds_bytes(v, bf16, ps[0]);
    for (int i = 1; i < count; i++) {
        if (!same_shape(ps[0], ps[i])) return hipErrorInvalidValue;
        g.m[i - 1] = ConvMember{ps[i].in, ps[i].in_R, ps[i].wp, ps[i].bias, ps[i].out,
                                ps[i].out_R, ps[i].res, ps[i].res_R, ps[i].k};
        const size_t l = conv_lds_bytes(v, bf16, ps[i]);
        lds = l > lds ? l : lds;
    }
    return bf16 ? launch_dt<true>(v, g, count, lds, st) : launch_dt<false>(v, g, count, lds, st);
}

// ------------------------------------------------------ fused resblock pair
//
// One block: one branch's pair at one dilation, for stream b and the frames
// [f0, f1) of its segment, all C channels, in sub-tiles of BM frames.  LDS
// holds two windows indexed by frame modulo their size:
//   Zs  LeakyReLU(z) as bf16 for the frames the first conv reads
//       ([t - (k-1)d - (k-1), t + BM) for the sub-tile at t), WZ = 2^LZ frames;
//   Hs  h = LeakyReLU(conv1 + b1) as bf16 ([t - (k-1), t + BM)), WH = 2^LH
//       frames; zero for frames before the stream's start, as a freshly reset
//       ring holds.
// Per sub-tile: the first conv writes h for its BM frames (the first sub-tile
// of the segment also the 16 frames left of it, of which the second conv reads
// the last k - 1); after a barrier the second conv reads Hs and the epilogue
// adds b2, the residual z and the branch mean; then the next sub-tile's
// BM z frames go to Zs, replacing frames older than any the next first conv
// reads.  Both convs use one K partition and a channel block of all C
// channels, i.e. the arithmetic of the unfused launches with those
// parameters, bit for bit.

template <int MB, int NB, int WGM, int WGN, int KCH, int LZ, int LH>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void pair_kernel(const PairGroup g)
{
    const PairParams& p = g.p;
    const uint16_t* z = p.z;
    int z_R = (int)p.z_R;
    const void* w1p = p.w1;
    const float* b1 = p.b1;
    const void* w2p = p.w2;
    const float* b2 = p.b2;
    uint16_t* out = p.out;
    int out_R = (int)p.out_R;
    int k = p.k;
    if (blockIdx.z > 0) {
        const PairMember& m = g.m[blockIdx.z - 1];
        z = m.z;
        z_R = (int)m.z_R;
        w1p = m.w1;
        b1 = m.b1;
        w2p = m.w2;
        b2 = m.b2;
        out = m.out;
        out_R = (int)m.out_R;
        k = m.k;
    }
    constexpr int KQ = 32;
    constexpr int C = KQ * KCH;
    constexpr int BM = 16 * MB * WGM, BN = 16 * NB * WGN;
    constexpr int LDW = C + OpT<true>::PAD;
    constexpr int VPR = C / 8;                 // 8-channel groups per frame
    constexpr int ZM = (1 << LZ) - 1, HM = (1 << LH) - 1;
    static_assert(WGM * WGN == 4 && BN == C, "pair tile shape");
    using Frag = u32x4;

    const int H1 = (k - 1) * p.d, H2 = k - 1, H = H1 + H2;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* Zs = reinterpret_cast<uint16_t*>(smem);
    uint16_t* Hs = Zs + (ZM + 1) * LDW;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WGM, wn = wave / WGM;
    const int b = blockIdx.x / p.segs;
    const int f0 = (blockIdx.x - b * p.segs) * p.seg_t * BM;
    const int f1 = min(p.F, f0 + p.seg_t * BM);
    const int64_t tau0 = p.clock[0] * p.in_fpt;
    const int64_t start_f = p.start[b] * p.in_fpt;   // this stream's first frame since its reset
    const int fl = lane & 15, cg = (lane >> 4) * 4;
    const uint16_t* zb = z + (size_t)b * z_R * C;
    const int zs0 = (int)ring_slot(tau0 + f0 - H, z_R);   // ring slot of frame f0 - H
    // ring slot of frame f of this chunk, for f0 - H <= f < f0 - H + z_R
    auto zslot = [&](int f) {
        DC_DBG_CHECK(b < p.B && f - (f0 - H) >= 0 && f - (f0 - H) < z_R, kDbgPairZ);
        return slot_add(zs0, f - (f0 - H), z_R);
    };

    // z frames [fa, fa + n) -> Zs (LeakyReLU, bf16); frames at or past F are
    // zeros.  A thread's vectors go SU at a time: their loads are all issued
    // before the first is converted (a vector past the range, or of a frame
    // at or past F, loads frame fa, which is in the ring).
    auto stage = [&](int fa, int n) {
        constexpr int SU = 8;
        for (int v0 = tid; v0 < n * VPR; v0 += 256 * SU) {
            u32x4 q[SU];
#pragma unroll
            for (int u = 0; u < SU; u++) {
                const int v = v0 + 256 * u, r = v / VPR, c8 = (v - r * VPR) * 8;
                const bool in = v < n * VPR && fa + r < p.F;
                q[u] = *(const u32x4*)(zb + (size_t)zslot(in ? fa + r : fa) * C + (in ? c8 : 0));
            }
            __builtin_amdgcn_sched_barrier(0);   // all loads before the first use
#pragma unroll
            for (int u = 0; u < SU; u++) {
                const int v = v0 + 256 * u, r = v / VPR, c8 = (v - r * VPR) * 8;
                const int f = fa + r;
                float x[8];
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    x[2 * e] = f < p.F ? lrelu(h2f(q[u][e] & 0xffffu), p.slope) : 0.f;
                    x[2 * e + 1] = f < p.F ? lrelu(h2f(q[u][e] >> 16), p.slope) : 0.f;
                }
                if (v < n * VPR) store8_lds(Zs + (f & ZM) * LDW + c8, x);
            }
        }
    };
    // the same for the BM frames of the next sub-tile in two halves: fetch
    // issues the loads (frames past F read frame F - 1, so every lane loads
    // and nothing waits on a branch), commit converts and writes Zs after
    // the second conv has run in their shadow.  At C = 128 the registers the
    // loads hold would spill: there the next frames are staged after the
    // epilogue instead.
    constexpr bool PF = KCH <= 2;
    constexpr int PV = BM * VPR / 256;
    static_assert(BM * VPR % 256 == 0, "pair staging vectors");
    auto fetch = [&](int fa, u32x4 (&q)[PV]) {
#pragma unroll
        for (int i = 0; i < PV; i++) {
            const int v = tid + 256 * i, r = v / VPR, c8 = (v - r * VPR) * 8;
            const int f = min(fa + r, p.F - 1);
            q[i] = *(const u32x4*)(zb + (size_t)zslot(f) * C + c8);
        }
    };
    auto commit = [&](int fa, const u32x4 (&q)[PV]) {
#pragma unroll
        for (int i = 0; i < PV; i++) {
            const int v = tid + 256 * i, r = v / VPR, c8 = (v - r * VPR) * 8;
            const int f = fa + r;
            float x[8];
#pragma unroll
            for (int e = 0; e < 4; e++) {
                x[2 * e] = f < p.F ? lrelu(h2f(q[i][e] & 0xffffu), p.slope) : 0.f;
                x[2 * e + 1] = f < p.F ? lrelu(h2f(q[i][e] >> 16), p.slope) : 0.f;
            }
            store8_lds(Zs + (f & ZM) * LDW + c8, x);
        }
    };
    // weight fragments of tap j (channel block of all C channels, one partition)
    const int nblk0 = wn * NB;
    // both convs' biases of this wave's columns, loaded once for the whole run
    f32x4 bias1[NB], bias2[NB];
#pragma unroll
    for (int nb = 0; nb < NB; nb++) {
        bias1[nb] = *(const f32x4*)(b1 + (nblk0 + nb) * 16 + cg);
        bias2[nb] = *(const f32x4*)(b2 + (nblk0 + nb) * 16 + cg);
    }
    auto load_tap = [&](const Frag* wp, int j, Frag (&w)[KCH][NB]) {
        const Frag* wt = wp + (size_t)j * KCH * p.NB16 * 64 + lane;
#pragma unroll
        for (int ki = 0; ki < KCH; ki++)
#pragma unroll
            for (int nb = 0; nb < NB; nb++) w[ki][nb] = wt[((size_t)ki * p.NB16 + nblk0 + nb) * 64];
    };
    // the taps of one conv in pairs, weights one tap ahead (as in conv_kernel);
    // `issued` runs once the first two taps' weight loads are issued
    auto run_taps = [&](const Frag* wp, auto&& tap, auto&& issued) {
        Frag w0[KCH][NB], w1[KCH][NB];
        load_tap(wp, 0, w0);
        if (k == 1) issued();
        int j = 0;
        for (; j + 1 < k; j += 2) {
            load_tap(wp, j + 1, w1);
            if (j == 0) issued();
            __builtin_amdgcn_sched_barrier(0);
            tap(j, w0);
            __builtin_amdgcn_sched_barrier(0);
            load_tap(wp, j + 2 < k ? j + 2 : j + 1, w0);
            __builtin_amdgcn_sched_barrier(0);
            tap(j + 1, w1);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (j < k) tap(j, w0);
    };
    const int koff = (lane >> 4) * 8;
    auto nothing = [] {};

    // first conv over R row blocks of 16 frames starting at frame fr (this
    // lane: frames fr + 16 i + fl); h -> Hs
    auto conv1 = [&](auto rb_tag, int fr) {
        constexpr int R = decltype(rb_tag)::value;
        f32x4 acc[R][NB];
#pragma unroll
        for (int i = 0; i < R; i++)
#pragma unroll
            for (int nb = 0; nb < NB; nb++) acc[i][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int row0 = fr + fl - H1;         // z frame of tap 0 for row block 0
        // a row block's frame fragment of the next channel chunk is read
        // right after that block's MFMAs of this chunk, into the same
        // registers: the read has the other row blocks' MFMAs to arrive in
        auto tap1 = [&](int j, const Frag (&w)[KCH][NB]) {
            int ai[R];
#pragma unroll
            for (int i = 0; i < R; i++) ai[i] = ((row0 + 16 * i + j * p.d) & ZM) * LDW + koff;
            bf16x8_t a[R];
#pragma unroll
            for (int i = 0; i < R; i++) a[i] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(Zs + ai[i]));
#pragma unroll
            for (int ki = 0; ki < KCH; ki++) {
#pragma unroll
                for (int i = 0; i < R; i++) {
#pragma unroll
                    for (int nb = 0; nb < NB; nb++)
                        acc[i][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[ki][nb]),
                                                                            a[i], acc[i][nb], 0, 0, 0);
                    if (ki + 1 < KCH)
                        a[i] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(Zs + ai[i] + (ki + 1) * KQ));
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        };
        run_taps(reinterpret_cast<const Frag*>(w1p), tap1, nothing);
#pragma unroll
        for (int i = 0; i < R; i++) {
            const int f = fr + 16 * i + fl;
            const bool before = tau0 + f < start_f;   // h of a frame before the stream start is 0
#pragma unroll
            for (int nb = 0; nb < NB; nb++) {
                f32x4 v = acc[i][nb] + bias1[nb];
#pragma unroll
                for (int e = 0; e < 4; e++) v[e] = before ? 0.f : lrelu(v[e], p.slope);
                typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;
                const u32x2 hv = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *(u32x2*)(Hs + (f & HM) * LDW + (nblk0 + nb) * 16 + cg) = hv;
            }
        }
    };

    const int mean_R = (int)p.mean_R;
    uint32_t f16_mag = 0;   // largest output magnitude's bits (checked once, at the end)
    stage(f0 - H, BM + H);
    __syncthreads();
    for (int t = f0; t < f1; t += BM) {
        // ---- first conv: h for this wave's rows of [t, t + BM) (and [t - 16, t) first)
        if (t == f0 && wm == 0)
            conv1(std::integral_constant<int, MB + 1>{}, t - 16);   // with the 16 frames left of the run
        else
            conv1(std::integral_constant<int, MB>{}, t + wm * 16 * MB);
        __syncthreads();
        // the epilogue's residual and branch-mean vectors: fp16, four channels
        // of one frame, loaded raw and converted where used (rows past the
        // run read its last frame and store nothing)
        auto tl_of = [&](int mb) {
            const int tl = wm * 16 * MB + mb * 16 + fl;
            return t + tl < f1 ? tl : f1 - 1 - t;
        };
        auto h4 = [](u32x2 w) {
            return f32x4{h2f(w[0] & 0xffffu), h2f(w[0] >> 16), h2f(w[1] & 0xffffu), h2f(w[1] >> 16)};
        };
        auto issue_z = [&](int mb, u32x2 (&q)[NB]) {
            const uint16_t* zr = zb + (size_t)zslot(t + tl_of(mb)) * C + nblk0 * 16 + cg;
#pragma unroll
            for (int nb = 0; nb < NB; nb++) q[nb] = *(const u32x2*)(zr + nb * 16);
        };
        // the next sub-tile's z frames (where registers allow) and, without a
        // branch mean, the residual, loaded while the second conv runs
        u32x4 zq[PV];
        u32x2 zpre[MB][NB];
        if constexpr (PF) {
            if (t + BM < f1) fetch(t + BM, zq);
        }
        if (p.n_mean == 0) {
#pragma unroll
            for (int mb = 0; mb < MB; mb++) issue_z(mb, zpre[mb]);
        }

        // ---- second conv: output frames t + wm*16*MB + 16 mb + fl, h from Hs
        f32x4 acc[MB][NB];
#pragma unroll
        for (int i = 0; i < MB; i++)
#pragma unroll
            for (int nb = 0; nb < NB; nb++) acc[i][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int hrow0 = t + wm * 16 * MB + fl - H2;
        // frame fragments are read one channel chunk ahead of their MFMAs
        auto tap2 = [&](int j, const Frag (&w)[KCH][NB]) {
            int hi[MB];
#pragma unroll
            for (int mb = 0; mb < MB; mb++) hi[mb] = ((hrow0 + 16 * mb + j) & HM) * LDW + koff;
            bf16x8_t a[2][MB];
#pragma unroll
            for (int mb = 0; mb < MB; mb++) a[0][mb] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(Hs + hi[mb]));
#pragma unroll
            for (int ki = 0; ki < KCH; ki++) {
                if (ki + 1 < KCH) {
#pragma unroll
                    for (int mb = 0; mb < MB; mb++)
                        a[(ki + 1) & 1][mb] = __builtin_bit_cast(bf16x8_t, *(const u32x4*)(Hs + hi[mb] + (ki + 1) * KQ));
                }
                __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of these MFMAs
#pragma unroll
                for (int mb = 0; mb < MB; mb++)
#pragma unroll
                    for (int nb = 0; nb < NB; nb++)
                        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w[ki][nb]),
                                                                             a[ki & 1][mb], acc[mb][nb], 0, 0, 0);
            }
        };
        run_taps(reinterpret_cast<const Frag*>(w2p), tap2, nothing);

        // ---- epilogue: bias, residual z, branch mean; fp16 through the output ring
        const int out_s = (int)ring_slot(tau0 + t, out_R);
        const int mean_s = p.n_mean ? (int)ring_slot(tau0 + t, p.mean_R) : 0;
        auto store = [&](int mb, int nb, f32x4 v) {
            const int tl = wm * 16 * MB + mb * 16 + fl;
            if (t + tl < f1)
                store4(out, kF16, ring_at(b, p.B, slot_add(out_s, tl, out_R), out_R, (nblk0 + nb) * 16 + cg, 4, C, kDbgPairOut),
                       v, &f16_mag);
        };
        if (p.n_mean == 0) {
            // the residual was loaded during the second conv
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++) store(mb, nb, h4(zpre[mb][nb]) + (acc[mb][nb] + bias2[nb]));
        } else {
            // with the branch means: every row block's residual and three mean
            // vectors are issued before the first is used (a mean past n_mean
            // reads the first and is not used, so the loads need no branch)
            const float J = (float)(p.n_mean + 1);
            const uint16_t* mp[3];
#pragma unroll
            for (int i = 0; i < 3; i++) mp[i] = p.mean[i < p.n_mean ? i : 0];
            u32x2 r[MB][NB], m[MB][3][NB];
#pragma unroll
            for (int mb = 0; mb < MB; mb++) {
                issue_z(mb, r[mb]);
                const size_t mo = ring_at(b, p.B, slot_add(mean_s, tl_of(mb), mean_R), mean_R, nblk0 * 16 + cg,
                                          (NB - 1) * 16 + 4, C, kDbgPairOut);
#pragma unroll
                for (int i = 0; i < 3; i++)
#pragma unroll
                    for (int nb = 0; nb < NB; nb++) m[mb][i][nb] = *(const u32x2*)(mp[i] + mo + nb * 16);
            }
#pragma unroll
            for (int mb = 0; mb < MB; mb++) {
#pragma unroll
                for (int nb = 0; nb < NB; nb++) {
                    const f32x4 v = h4(r[mb][nb]) + (acc[mb][nb] + bias2[nb]);
                    f32x4 x = h4(m[mb][0][nb]);
                    if (p.n_mean > 1) x = x + h4(m[mb][1][nb]);
                    if (p.n_mean > 2) x = x + h4(m[mb][2][nb]);
                    x = x + v;
                    store(mb, nb, f32x4{x[0] / J, x[1] / J, x[2] / J, x[3] / J});
                }
            }
        }
        // the next sub-tile's z frames to Zs (the frames they replace are
        // older than any the next first conv reads)
        if (t + BM < f1) {
            if constexpr (PF)
                commit(t + BM, zq);
            else
                stage(t + BM, BM);
        }
        __syncthreads();
    }
    raise_f16_range(p.err, f16_mag);
}

// Fused-pair shapes (ids of this table).
static const PairShape kPairs[] = {
    // MB NB WGM WGN KCH LZ LH
    {2, 2, 2, 2, 2, 7, 7},   // 0: C = 64, 64-frame sub-tiles
    {4, 2, 2, 2, 2, 8, 8},   // 1: C = 64, 128-frame sub-tiles
    {4, 2, 1, 4, 4, 7, 7},   // 2: C = 128, 64-frame sub-tiles
};

int num_pair_variants() { return (int)(sizeof(kPairs) / sizeof(kPairs[0])); }
PairShape pair_variant(int v) { return kPairs[v]; }

size_t pair_lds_bytes(int v)
{
    const PairShape& t = kPairs[v];
    return (size_t)(t.WZ() + t.WH()) * (t.C() + OpT<true>::PAD) * 2;
}

template <int MB, int NB, int WGM, int WGN, int KCH, int LZ, int LH>
static hipError_t launch_pair_t(const PairGroup& g, int count, size_t lds, hipStream_t st)
{
    const PairParams& p = g.p;
    dim3 grid((unsigned)(p.B * p.segs), 1u, (unsigned)count);
    static size_t lds_set[kMaxDevices] = {};
    const hipError_t e = allow_lds(reinterpret_cast<const void*>(&pair_kernel<MB, NB, WGM, WGN, KCH, LZ, LH>), lds,
                                   lds_set);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((pair_kernel<MB, NB, WGM, WGN, KCH, LZ, LH>), grid, dim3(256), lds, st, g);
    return hipGetLastError();
}

hipError_t launch_pair(int v, const PairParams* ps, int count, hipStream_t st)
{
    if (count < 1 || count > kMaxGroup || v < 0 || v >= num_pair_variants()) return hipErrorInvalidValue;
    const PairShape t = kPairs[v];
    PairGroup g{};
    g.p = ps[0];
    for (int i = 0; i < count; i++) {
        const PairParams& a = ps[0];
        const PairParams& q = ps[i];
        if (q.d != a.d || q.C != a.C || q.NB16 != a.NB16 || q.B != a.B || q.F != a.F || q.tiles_t != a.tiles_t ||
            q.seg_t != a.seg_t || q.segs != a.segs || q.n_mean != a.n_mean || q.clock != a.clock ||
            q.start != a.start || q.in_fpt != a.in_fpt || q.slope != a.slope || !t.fits(q.k, q.d))
            return hipErrorInvalidValue;
        if (i > 0) g.m[i - 1] = PairMember{q.z, q.z_R, q.w1, q.b1, q.w2, q.b2, q.out, q.out_R, q.k};
    }
    const PairParams& p = ps[0];
    if (p.C != t.C() || p.tiles_t != (p.F + t.BM() - 1) / t.BM() || p.seg_t < 1 ||
        (int64_t)p.segs * p.seg_t < p.tiles_t || (int64_t)(p.segs - 1) * p.seg_t >= p.tiles_t)
        return hipErrorInvalidValue;
    const size_t lds = pair_lds_bytes(v);
    switch (v) {
    case 0: return launch_pair_t<2, 2, 2, 2, 2, 7, 7>(g, count, lds, st);
    case 1: return launch_pair_t<4, 2, 2, 2, 2, 8, 8>(g, count, lds, st);
    case 2: return launch_pair_t<4, 2, 1, 4, 4, 7, 7>(g, count, lds, st);
    default: return hipErrorInvalidValue;
    }
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
    const size_t dst = ring_at(b, B, slot, out.R, c8, 8, C, kDbgEmbed);
    const bool ok = tok >= 0 && tok < vocab;
    if (!ok) *err = kErrTokenId;
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
//
// The tables fold the real inverse DFT, the periodic Hann window and the
// overlap-add normaliser (computed in double on the host from their
// definitions): g[n] = sum_kk Tre[n][kk] Re X_kk + Tim[n][kk] Im X_kk with
// X_kk = exp(logmag_kk) (cos ph_kk + i sin ph_kk).  A windowed frame's zeroed
// ring slot stands for a frame before the start of the stream.
constexpr int kNFFT = 16, kBins = 9;

// ----------------------------------------------- iSTFT tail, one kernel
//
// Spectrum, inverse DFT, window and overlap-add of one call in one launch.  A
// block owns kTail consecutive frames [f0, f0 + kTail) of one stream: each
// thread turns one frame's log-magnitude and phase into its windowed frame g
// in LDS (exp and sincos per bin, then per output sample a chain of fmas over
// the bins in ascending order, real part before imaginary), where the block
// also holds the 3 frames before f0 -- recomputed from the head output when
// they belong to this call, read from the G ring when they are the previous
// call's.  Then each thread overlap-adds the hop = 4 samples of its frame
// from the LDS rows of the 4 frames that cover them, in ascending frame order
// starting from +0, and stores them as one vector.  Only the call's last 3
// frames go to the G ring: they are the next call's left context.  Every
// sample's arithmetic depends only on its frame index, so a frame gives the
// same bits in any block, call or chunking.
//
// The launch also ends the call: with `advance` set, the last block to finish
// adds the call's tokens to the device clock.  Every block counts itself in
// `arrivals` after its last read of the clock, so the block that counts last
// knows that no block still reads the old value; it then re-arms the count
// for the next call.
//
// kTail + 3 = 256: every thread builds exactly one LDS row, so no thread
// runs the per-frame chain (head loads, exp and sincos, the fmas) twice.
constexpr int kTail = 253;

__global__ __launch_bounds__(256) void istft_kernel(const float* head, int64_t head_R, int B, int F,
                                                    const float* table, Ring g, float* pcm,
                                                    int64_t* clock, int64_t fpt, int n_advance,
                                                    unsigned* arrivals)
{
    constexpr int W = kNFFT + 1;                 // LDS row stride (odd: no bank conflicts)
    __shared__ float G[(kTail + 3) * W];
    const int tiles = (F + kTail - 1) / kTail;
    const int b = blockIdx.x / tiles, f0 = (blockIdx.x - b * tiles) * kTail;
    const int64_t tau0 = clock[0] * fpt;          // absolute index of this call's frame 0
    for (int i = threadIdx.x; i < kTail + 3; i += blockDim.x) {
        const int m = f0 - 3 + i;                 // frame of this call (negative: the previous call's)
        if (m >= F) continue;
        float* row = G + i * W;
        const int64_t tau = tau0 + m;
        if (m < 0) {
            const float* src = (const float*)g.ptr + ring_at(b, B, ring_slot(tau, g.R), g.R, 0, kNFFT, kNFFT, kDbgTail);
#pragma unroll
            for (int k = 0; k < kNFFT; k++) row[k] = src[k];
            continue;
        }
        // the frame's 2 * kBins values: 8-byte aligned, so loaded as pairs
        typedef __attribute__((ext_vector_type(2))) float f32x2;
        const f32x2* sp2 = (const f32x2*)(head + ring_at(b, B, ring_slot(tau, head_R), head_R, 0, 2 * kBins,
                                                          2 * kBins, kDbgTail));
        float sp[2 * kBins];
#pragma unroll
        for (int j = 0; j < kBins; j++) {
            const f32x2 q = sp2[j];
            sp[2 * j] = q[0];
            sp[2 * j + 1] = q[1];
        }
        float re[kBins], im[kBins];
#pragma unroll
        for (int kk = 0; kk < kBins; kk++) {
            const float mag = expf(sp[kk]);
            float sn, cs;
            sincosf(sp[kBins + kk], &sn, &cs);
            re[kk] = mag * cs;
            im[kk] = mag * sn;
        }
#pragma unroll
        for (int n = 0; n < kNFFT; n++) {
            const float* tr = table + n * kBins;
            const float* ti = table + kNFFT * kBins + n * kBins;
            float v = 0.f;
#pragma unroll
            for (int kk = 0; kk < kBins; kk++) {
                v = fmaf(tr[kk], re[kk], v);
                v = fmaf(ti[kk], im[kk], v);
            }
            row[n] = v;
        }
        if (m >= F - 3 && i >= 3) {               // the next call's left context
            float* dst = (float*)g.ptr + ring_at(b, B, ring_slot(tau, g.R), g.R, 0, kNFFT, kNFFT, kDbgTail);
#pragma unroll
            for (int n4 = 0; n4 < kNFFT; n4 += 4)
                *(f32x4*)(dst + n4) = f32x4{row[n4], row[n4 + 1], row[n4 + 2], row[n4 + 3]};
        }
    }
    __syncthreads();
    const int t = threadIdx.x, m = f0 + t;
    if (t < kTail && m < F) {
        // samples 4m + r: frames m - 3 + q (q = 0..3) at offset 12 - 4q + r
        f32x4 o;
#pragma unroll
        for (int r = 0; r < 4; r++) {
            float acc = 0.f;
#pragma unroll
            for (int q = 0; q < 4; q++) acc = acc + G[(t + q) * W + 12 - 4 * q + r];
            o[r] = acc;
        }
        *(f32x4*)(pcm + ring_at(b, B, m, F, 0, 4, 4, kDbgTail)) = o;
    }
    if (n_advance > 0) {
        __syncthreads();   // every thread of this block is past its use of the clock
        if (threadIdx.x == 0) {
            __threadfence();
            const unsigned before = atomicAdd(arrivals, 1u);
            if (before + 1 == gridDim.x) {
                atomicAdd((unsigned long long*)clock, (unsigned long long)n_advance);
                atomicExch(arrivals, 0u);
            }
        }
    }
}

hipError_t launch_istft(const float* head, int64_t head_R, int B, int F, const float* table, Ring g, float* pcm,
                        int64_t* clock, int64_t fpt, int n_advance, unsigned* arrivals, hipStream_t st)
{
    const int tiles = (F + kTail - 1) / kTail;
    hipLaunchKernelGGL(istft_kernel, dim3((unsigned)(B * tiles)), dim3(256), 0, st, head, head_R, B, F, table, g,
                       pcm, clock, fpt, n_advance, arrivals);
    return hipGetLastError();
}

// ------------------------------------------------ harmonic-plus-noise source
//
// The vocoder's stochastic input: sinusoids at the fundamental f0 and its
// overtones plus Gaussian noise, merged by a linear layer and tanh.  Every
// random number is a function of a counter -- the sample index since the
// stream's start -- so replayed, direct, chunked and offline decodes draw the
// same values (Design, clause (iii): the device generator advances along a
// declared clock; here the clock is the stream's own sample clock rather than
// the call count, which also makes the draws independent of the chunking).

// Philox4x64-10 and to_u01: dc_philox.h.

// Phase of each sinusoid at the start of every frame of this call, carried
// across calls: one thread per (stream, sinusoid) walks the frames in order,
// P <- frac(P + S * (h+1) f0 / sr), the fp64 operations of an offline walk.
// A stream at its first frame starts from its initial phase (0 for the
// fundamental, a draw of counter (0, h, 1, 0) for overtone h).  The carry
// has two slots tagged with the f0 frame they hold: a call reads the slot of
// its first frame and writes the other, so running a call's launch again
// reproduces it (the carry of a stream is never overwritten in place).
__global__ __launch_bounds__(64) void phase_kernel(const SourceParams p)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= p.B * p.H1) return;
    const int b = i / p.H1, h = i - (i / p.H1) * p.H1;
    const int64_t first = p.clock[0] * p.fpt0;              // f0 frame of this call's start
    const int sel = p.tags[2 * b] == first ? 0 : 1;
    double P = p.carry[((size_t)b * 2 + sel) * p.H1 + h];
    if (p.clock[0] == p.start[b]) {
        P = 0.0;
        if (h > 0) P = to_u01(philox4x64_10(0, (uint64_t)h, 1, 0, p.seed, p.keys[b]).v[0]);
    }
    const float* f0 = p.f0 + (size_t)b * p.F0;
    double* pt = p.ptab + (size_t)b * p.F0 * p.H1 + h;
    for (int f = 0; f < p.F0; f++) {
        pt[(size_t)f * p.H1] = P;
        const double inc = (double)(h + 1) * (double)f0[f] / p.sr;
        const double x = P + (double)p.S * inc;
        P = x - floor(x);
    }
    p.carry[((size_t)b * 2 + 1 - sel) * p.H1 + h] = P;
    if (h == 0) p.tags[2 * b + 1 - sel] = first + p.F0;   // (the slot read above keeps its tag)
}

hipError_t launch_phase(const SourceParams& p, hipStream_t st)
{
    const int n = p.B * p.H1;
    hipLaunchKernelGGL(phase_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, st, p);
    return hipGetLastError();
}

// One thread per (stream, sample of this call).  Sample t of the call lies
// in f0 frame t / S at offset r; its
// sinusoid h has phase frac(P_h[frame] + (r+1) (h+1) f0 / sr).  Noise of
// sinusoids 4g .. 4g+3 comes from Philox4x64-10 with key (seed, stream) and
// counter (sample since the stream's start, g, 0, 0), by Box-Muller on its
// draws (0, 1) and (2, 3).  src = tanh(mb + sum_h mw[h] e_h), h ascending.
// The stream's key is keys[b]: its index, unless its carry was imported from
// another slot (dc_carry_import), whose key it keeps.
constexpr int kMaxSinusoids = 32;

__global__ __launch_bounds__(256) void source_kernel(const SourceParams p)
{
    // (a sample's draws and sinusoids are independent of its neighbours';
    // four consecutive lanes write one last-stage frame's four samples)
    const int FL = p.F0 / (int)p.fpt0 * (int)p.fptL;   // last-stage frames of this call
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)p.B * FL * 4) return;
    const int b = (int)(i / (4 * FL)), t = (int)(i - (i / (4 * FL)) * (4 * FL));   // sample of this call
    const int tau = t >> 2, j = t & 3;
    const int64_t tauL = p.clock[0] * p.fptL + tau;                  // absolute last-stage frame
    const int64_t t_rel = (tauL - p.start[b] * p.fptL) * 4 + j;     // sample index since the stream's start
    const float* f0 = p.f0 + (size_t)b * p.F0;
    const double* ptab = p.ptab + (size_t)b * p.F0 * p.H1;
    const int groups = (p.H1 + 3) / 4;
    const uint64_t key = p.keys[b];
    const int f = t / p.S, r = t - (t / p.S) * p.S;
    const float fv = f0[f];
    const bool voiced = fv > p.thr;
    const float nscale = voiced ? p.noise : p.amp / 3.0f;
    float acc = 0.f;
    for (int g = 0; g < groups; g++) {
        const Philox4 x = philox4x64_10((uint64_t)t_rel, (uint64_t)g, 0, 0, p.seed, key);
        float nz[4];
#pragma unroll
        for (int q = 0; q < 2; q++) {
            const float rad = (float)sqrt(-2.0 * log(to_u01(x.v[2 * q])));
            const float ang = (float)(2.0 * M_PI * to_u01(x.v[2 * q + 1]));
            float sn, cs;
            sincosf(ang, &sn, &cs);
            nz[2 * q] = rad * cs;
            nz[2 * q + 1] = rad * sn;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int h = 4 * g + q;
            if (h >= p.H1) break;
            const double inc = (double)(h + 1) * (double)fv / p.sr;
            const double ph = ptab[(size_t)f * p.H1 + h] + (double)(r + 1) * inc;
            const float frac = (float)(ph - floor(ph));
            const float sine = voiced ? p.amp * sinf(6.28318530717958647692f * frac) : 0.f;
            acc = acc + p.mw[h] * (sine + nz[q] * nscale);
        }
    }
    p.src[((size_t)b * p.src_R + ring_slot(tauL, p.src_R)) * 4 + j] = tanhf(p.mb[0] + acc);
}

hipError_t launch_source(const SourceParams& p, hipStream_t st)
{
    const int64_t n = (int64_t)p.B * (p.F0 / p.fpt0 * p.fptL) * 4;
    hipLaunchKernelGGL(source_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p);
    return hipGetLastError();
}

// --------------------------------------------------------- stream starts

// start[b] = the clock minus `back` tokens (in stream order): stream b
// restarted `back` tokens before the next call; keys[b] keys its source
// generator.
__global__ void mark_start_kernel(int64_t* start, uint64_t* keys, int b, const int64_t* clock, int64_t back,
                                  uint64_t key)
{
    if (threadIdx.x == 0) {
        start[b] = clock[0] - back;
        keys[b] = key;
    }
}

hipError_t launch_mark_start(int64_t* start, uint64_t* keys, int b, const int64_t* clock, int64_t back, uint64_t key,
                             hipStream_t st)
{
    hipLaunchKernelGGL(mark_start_kernel, dim3(1), dim3(64), 0, st, start, keys, b, clock, back, key);
    return hipGetLastError();
}

// keys[b] = b: every stream keys its source generator with its own index.
__global__ void init_keys_kernel(uint64_t* keys, int B)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < B) keys[i] = (uint64_t)i;
}

hipError_t launch_init_keys(uint64_t* keys, int B, hipStream_t st)
{
    hipLaunchKernelGGL(init_keys_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, st, keys, B);
    return hipGetLastError();
}

}  // namespace dc

// Bounds-check bits of a checked build (see ring_at); -1 in a release build.
extern "C" int32_t dc_debug_checks(int32_t clear)
{
#ifdef DC_DEBUG
    int bits[64];
    if (hipDeviceSynchronize() != hipSuccess) return -2;
    if (hipMemcpyFromSymbol(bits, HIP_SYMBOL(dc::dc_debug_bits), sizeof(bits)) != hipSuccess) return -2;
    int all = 0;
    for (int i = 0; i < 64; i++) all |= bits[i];
    if (clear) {
        const int zero[64] = {0};
        if (hipMemcpyToSymbol(HIP_SYMBOL(dc::dc_debug_bits), zero, sizeof(zero)) != hipSuccess) return -2;
    }
    return all;
#else
    (void)clear;
    return -1;
#endif
}
