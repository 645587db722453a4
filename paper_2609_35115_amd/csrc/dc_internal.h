// Internal interface between the host runtime (dc_runtime.hip) and the gfx950
// kernels (dc_kernels.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dc {

// Element type of a ring buffer or of a conv operand.  kF16 (IEEE binary16)
// holds the fp32-accumulated residual stream of a bf16 decoder: values of
// order one keep 11 significant bits at half the bytes of fp32.
enum Elem : int { kF32 = 0, kBF16 = 1, kF16 = 2 };

// Bits of a state's device error flag (dc_sync reports and clears none of
// them; dc_reset clears them): a token id outside [0, vocab) reached the
// embedding, or a value that binary16 cannot hold (|v| >= 65520, which rounds
// to infinity, or NaN) was about to be stored in a bf16 state's residual stream.
enum ErrBit : int { kErrTokenId = 1, kErrF16Range = 2 };

inline int elem_bytes(int e) { return e == kF32 ? 4 : 2; }

// A ring of frames for B streams: frame with absolute index tau of stream b
// lives at ptr + ((b * R) + (tau mod R)) * C elements.  R >= ctx + frames of
// the largest call, so a call's frames never overwrite the left context
// (ctx frames) its consumers read.
struct Ring {
    void* ptr = nullptr;
    int C = 0;
    int elem = kF32;
    int64_t R = 0;
    int ctx = 0;
    int level = 0;          // clock level: 0 = pre-stack frames, s+1 = after stage s
};

// One implicit-GEMM causal convolution launch.
//   rows   (b, t): stream b, frame t in [0, F) of this call (input clock)
//   cols   n in [0, N)
//   K      (channel block cb, tap j, channel c): fixed order, independent of
//          every launch parameter except the layer's own geometry
//   out    conv:  frame t, channel n
//          convT: frame t*u + n / Co, channel n % Co  (polyphase transposed conv)
struct ConvParams {
    const void* in;
    int64_t in_R;
    int in_C;
    int in_elem;
    int in_act;           // apply LeakyReLU to the operand at load
    int split;            // bf16 only: operand as hi + lo bf16 pair (two MFMAs per step)
    const void* wp;       // packed weights, operand element type
    const float* bias;    // [N]
    int CB;               // channels per block (multiple of the MFMA K quantum)
    int n_cb;             // channel blocks (CB * n_cb >= in_C, zero padded)
    int k, d;             // taps, dilation
    int N;                // real columns
    int NB16;             // packed column blocks of 16
    void* out;
    int64_t out_R;
    int out_C;
    int out_elem;
    int out_act;          // apply LeakyReLU before the store
    int u;                // 1 for a conv, stride u for a transposed conv
    const void* res;      // residual ring (element type out_elem, out geometry) or null
    int64_t res_R;
    const void* mean[3];  // earlier branch results (rings of element type out_elem, out geometry)
    int64_t mean_R;
    int n_mean;           // >0: out = (mean[0] + ... + mean[n_mean-1] + z) / (n_mean + 1)
    int B, F;             // streams, input frames of this call
    int tiles_t;          // ceil(F / BM)
    const int64_t* clock; // tokens decoded before this call
    int64_t in_fpt;       // input-clock frames per token
    float slope;
    // harmonic source (the last stage's ConvTranspose1d only, else null):
    // out[frame][c] += sd_b[c] + sum_j sd_w[c][j] * src[frame][j], src a ring
    // of 4 samples per output frame (out geometry)
    const float* src;
    int64_t src_R;
    const float* sd_w;    // [out_C][4]
    const float* sd_b;    // [out_C]
    int* err;             // the state's device error flag (kErrF16Range on a binary16 overflow)
};

// Block of 4 waves: WGM x WGN waves tile the output, each wave MB x NB MFMA
// blocks of 16x16; WGK waves split K (each takes every WGK-th K chunk of a
// tap).  KCH is the channel block in MFMA K chunks.  WGK and KCH are part of
// a layer's arithmetic (they fix the order of the fp32 sums); MB, NB, WGM,
// WGN and W (how weight fragments reach the waves) are not.
// One launch runs the same tile shape over up to kMaxGroup convs that differ
// only in taps, weights, bias and their input, output and residual rings
// (the parallel branches of a resblock stage): blockIdx.z selects the member.
// Member 0 is a full parameter set; the others carry only what differs, so
// every shared field stays at a fixed kernel-argument offset.
constexpr int kMaxGroup = 4;
struct ConvMember {
    const void* in;
    int64_t in_R;
    const void* wp;
    const float* bias;
    void* out;
    int64_t out_R;
    const void* res;
    int64_t res_R;
    int k;
};
struct ConvGroup {
    ConvParams p;                      // member 0
    ConvMember m[kMaxGroup - 1];       // members 1..count-1
};

struct TileShape {
    int MB, NB, WGM, WGN, WGK, KCH;
    int W = 0;   // 1: weights through an LDS ring shared by the block's waves (bf16, WGK = 1)
    int BM() const { return 16 * MB * WGM; }
    int BN() const { return 16 * NB * WGN; }
    int S() const { return WGK; }
};

// One fused resblock pair (bf16 operands, fp16 residual stream):
// h = LeakyReLU(conv_k,d(LeakyReLU(z)) + b1) stays in LDS, and out = z + conv_k,1(h) + b2 (optionally averaged with
// earlier branch results).  A block owns one stream's frames
// [seg * seg_t * BM, (seg + 1) * seg_t * BM) x all C channels and walks them
// in sub-tiles of BM frames, keeping LeakyReLU(z) and h in LDS windows that
// slide with the sub-tile: the first sub-tile computes the k - 1 frames of h
// left of the run, later ones only their own BM frames.
struct PairParams {
    const uint16_t* z;    // fp16 ring: the first conv's input and the residual
    int64_t z_R;
    const void* w1;       // packed like a conv with channel block C (one partition)
    const float* b1;
    const void* w2;
    const float* b2;
    uint16_t* out;        // fp16 ring
    int64_t out_R;
    int k, d;             // taps; dilation of the first conv (the second has 1)
    int C;                // channels in and out of both convs
    int NB16;             // C / 16
    const uint16_t* mean[3]; // earlier branch results (fp16 rings, out geometry)
    int64_t mean_R;
    int n_mean;
    int B, F, tiles_t;    // tiles_t = ceil(F / BM) sub-tiles per stream
    int seg_t, segs;      // sub-tiles per block, blocks per stream (segs * seg_t >= tiles_t)
    const int64_t* clock;
    const int64_t* start; // [B]: tokens decoded when each stream last started
    int64_t in_fpt;
    float slope;
    int* err;             // the state's device error flag (kErrF16Range on a binary16 overflow)
};
struct PairMember {
    const uint16_t* z;
    int64_t z_R;
    const void* w1;
    const float* b1;
    const void* w2;
    const float* b2;
    uint16_t* out;
    int64_t out_R;
    int k;
};
struct PairGroup {
    PairParams p;
    PairMember m[kMaxGroup - 1];
};

// Fused-pair shapes: MB x NB blocks of 16x16 per wave (both convs), WGM x WGN
// waves, channel block KCH chunks (C = 32 KCH); LDS windows of 2^LZ frames of
// LeakyReLU(z) (>= BM + (k-1)(d+1)) and 2^LH frames of h (>= BM + 16).
struct PairShape {
    int MB, NB, WGM, WGN, KCH, LZ, LH;
    int BM() const { return 16 * MB * WGM; }
    int C() const { return 32 * KCH; }
    int WZ() const { return 1 << LZ; }
    int WH() const { return 1 << LH; }
    bool fits(int k, int d) const { return WZ() >= BM() + (k - 1) * (d + 1) && WH() >= BM() + 16 && k - 1 <= 16; }
};
int num_pair_variants();
PairShape pair_variant(int v);
size_t pair_lds_bytes(int v);
hipError_t launch_pair(int v, const PairParams* ps, int count, hipStream_t st);

// The tile shapes compiled for each operand type.
int num_tile_variants();
TileShape tile_variant(int v);

// LDS bytes a conv launch needs with tile shape v.
size_t conv_lds_bytes(int v, bool bf16, const ConvParams& p);

// LDS bytes of a launch of `count` convs (the largest member).
hipError_t launch_conv(int v, bool bf16, const ConvParams* ps, int count, hipStream_t st);

hipError_t launch_embed(const int32_t* tokens, int n, int B, const void* table, int vocab, int C,
                        int elem, int fpt, Ring out, const int64_t* clock, int* err, hipStream_t st);

// Head output -> PCM [B][F*hop] in one launch (spectrum, iDFT, window and
// overlap-add; n_fft = 16, hop = 4); writes the call's last 3 windowed frames
// to the G ring (the next call's left context) and reads the previous call's.
// With n_advance > 0 the launch also advances the clock by n_advance tokens
// once every block has read it (arrivals: a zeroed counter it leaves zeroed);
// 0 leaves the clock as it is (a launch re-run for timing).
hipError_t launch_istft(const float* head, int64_t head_R, int B, int F, const float* table, Ring g, float* pcm,
                        int64_t* clock, int64_t fpt, int n_advance, unsigned* arrivals, hipStream_t st);

// Harmonic-plus-noise excitation source of one call.
struct SourceParams {
    const float* f0;       // [B][F0] Hz per frame of the pre-stack clock (this call)
    double* carry;         // [B][2][H1] phase (cycles) at a frame start, two tagged slots
    int64_t* tags;         // [B][2] the f0 frame each slot's phases belong to
    double* ptab;          // [B][F0][H1] phase at the start of each frame of this call
    float* src;            // ring [B][src_R][4]: the samples of each last-stage frame
    int64_t src_R;
    const float* mw;       // merge weights [H1]
    const float* mb;       // merge bias [1]
    int B, F0, H1;         // streams, frames of this call, sinusoids (fundamental + overtones)
    int S;                 // samples per f0 frame
    int64_t fpt0, fptL;    // f0 frames and last-stage frames per token
    const int64_t* clock;
    const int64_t* start;  // [B] tokens decoded when each stream last started
    const uint64_t* keys;  // [B] each stream's generator key (second key word)
    float amp, noise, thr;
    double sr;
    uint64_t seed;
};
hipError_t launch_phase(const SourceParams& p, hipStream_t st);
hipError_t launch_source(const SourceParams& p, hipStream_t st);

hipError_t launch_mark_start(int64_t* start, uint64_t* keys, int b, const int64_t* clock, int64_t back, uint64_t key,
                             hipStream_t st);
hipError_t launch_init_keys(uint64_t* keys, int B, hipStream_t st);

}  // namespace dc
