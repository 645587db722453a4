// Internal interface between the flow-decoder runtime (flow_runtime.hip) and
// its gfx950 kernels (flow_kernels.hip).  Not part of the ABI.
//
// Rows of a call: stream b' in [0, Bc) of the call (stream b0 + b' of the
// state), guidance branch c (0 conditional, 1 unconditional), frame f in
// [0, n): row = (b' * 2 + c) * n + f.
//
// Carry of stream b: for every (solver step i, block l, branch c, kv, head)
// a region of Fr frames -- the prompt's frames at [0, Pr), then R + 1 slots
// of Sl frames at Pr + slot * Sl, slot = (retained chunks since the turn
// start) mod (R + 1), R = f_retained / f_chunk.  A call writes its own
// frames into the slot after the R newest, so the history it attends to is
// never overwritten while it runs, and a retained chunk is never moved.
// Keys are stored [frame][64]; values transposed [64][frame], the operand
// order of the attention's second product.  Region index:
//   ((((b * NS + i) * NL + l) * 2 + c) * 2 + kv) * heads + head.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcf {

// Calls of at most this many rows (2 per stream and frame) run the skinny GEMM.
constexpr int kSkinnyRows = 512;

enum Epi : int {
    E_H = 0,     // h = acc + bias                        (fp32)
    E_QKV = 1,   // q -> q buffer, k, v -> the carry      (operand type)
    E_RES = 2,   // h += gate * (acc + bias)              (fp32)
    E_GELU = 3,  // out = GELU_tanh(acc + bias)           (operand type)
    E_VEL = 4,   // out = acc + bias                      (fp32)
};

struct CarryRef {
    void* base;              // stream 0, step i, block l
    int64_t stream_stride;   // elements between streams
    int Fr;                  // frames per region
    int Pr, Sl, R;           // prompt frames, slot frames, history slots
    const int64_t* hist;     // [B] chunks retained since the turn start
    const int* plen;         // [B] prompt frames of the turn
};

// out[row][col] = epilogue(sum_k A[row][k] W[col][k] + bias[col]); with
// ln_h set, A[row][k] = LN(ln_h[row])[k] * (1 + ln_scale[k]) + ln_shift[k]
// (the modulated LayerNorm of the fp32 residual stream, K <= 512): normalised
// while staged for calls of few rows, else written to A by a launch of its own.
struct GemmParams {
    const void* A;           // [M][K] operand type (with ln_h: where the normalised operand may be written)
    const float* ln_h;       // [M][K] or null
    const float* ln_shift;   // [K]
    const float* ln_scale;   // [K]
    const void* W;           // [N][K] operand type
    const float* bias;       // [N]
    int M, N, K;
    float* h;                // E_H, E_RES: [M][N]
    const float* gate;       // E_RES: [N]
    void* out;               // E_GELU (operand type), E_VEL (fp32): [M][N]
    void* q;                 // E_QKV: [Bc][2][heads][Fq][64]
    int Fq;
    CarryRef carry;
    int prompt;              // 1: own frames go to the prompt region
    int n, b0, heads, dim;
};

struct AttnParams {
    const void* q;           // [Bc][2][heads][Fq][64]
    int Fq;
    CarryRef carry;
    void* o;                 // [M][dim] operand type
    int prompt;              // 1: the keys are the call's own frames only
    int n, b0, heads, dim, f_chunk;
};

struct AssembleParams {
    const float* mu;         // [Bc][n][n_mel]
    const float* cond;       // [Bc][n][n_mel] or null (zeros)
    const float* spk;        // [B][n_mel]
    float* x;                // [Bc][n][n_mel] solver state
    void* xin;               // [M][4 n_mel] operand type
    const int64_t* pos;      // [B] frame index since the turn start of the call's first frame
    const uint64_t* keys;    // [B] noise key of each stream
    uint64_t seed;
    float temperature;
    int n, b0, Bc, n_mel;
};

struct EulerParams {
    const float* v;          // [M][n_mel] estimator output
    float* x;                // [Bc][n][n_mel]
    void* xin;               // [M][4 n_mel]: x columns refreshed for the next step
    float* mel;              // [Bc][n][n_mel] on the last step, else null
    const float* dt;         // t_{i+1} - t_i
    float w;
    int n, Bc, n_mel;
};

struct ConstParams {
    const float* W1; const float* b1;   // time MLP
    const float* W2; const float* b2;
    const float* ada;                   // block 0's ada.W; blocks are ada_stride floats apart
    int64_t ada_stride;
    const float* fada;                  // final ada.W [2 dim][dim] then its bias
    float* silu_temb;                   // [NS][dim]
    float* mods;                        // [NS][NL][6 dim]
    float* fmods;                       // [NS][2 dim]
    float* t;                           // [NS + 1]
    float* dt;                          // [NS]
    int NS, NL, dim, t_dim;
};

hipError_t launch_consts(const ConstParams& p, hipStream_t st);
hipError_t launch_assemble(const AssembleParams& p, int bf16, hipStream_t st);
hipError_t launch_gemm(const GemmParams& p, int epi, int bf16, hipStream_t st);
hipError_t launch_attn(const AttnParams& p, int Bc, int bf16, hipStream_t st);
hipError_t launch_euler(const EulerParams& p, int bf16, hipStream_t st);
// Per-stream state: mode 0 begins a turn of stream b (no history, position
// 0, no prompt), mode 1 ends its prompt pass (position and prompt = P),
// mode 2 advances every stream by one retained chunk.
hipError_t launch_advance(int64_t* hist, int64_t* pos, int* plen, int mode, int b, int P, int B, int f_chunk,
                          hipStream_t st);
// The carry of (stream b, branch, kv) at the step and block of c.base in
// Eq. carry's logical order, widened to fp32: out [frames][heads * 64].
hipError_t launch_carry_gather(const CarryRef& c, int b, int branch, int kv, int heads, int bf16, int frames,
                               int f_chunk, float* out, hipStream_t st);

}  // namespace dcf
