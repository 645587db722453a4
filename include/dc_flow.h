/*
 * dc_flow.h — C ABI of the MI355X streaming flow-decoder chunk step.
 *
 * The flow decoder is the stage of the Token2Wav pipeline before the vocoder:
 * it turns the token encoder's features mu (n_mel values per frame) into mel
 * frames by conditional flow matching.  One call integrates dx/dt = v(x, t)
 * from Gaussian noise at t = 0 to t = 1 in n_steps explicit Euler steps on a
 * cosine time grid; v is the classifier-free-guided combination
 * (1 + w) v_cond - w v_uncond of a DiT estimator evaluated on the conditional
 * input (x | mu | speaker | prompt mel) and the unconditional one (x | 0 | 0 |
 * 0) (Motivation, "Where the time goes": a CFM solve with CFG x2 per second
 * of speech; Design, "Adapter": n_steps = 10).  Each attention of each block
 * at each solver step also attends to that step's carry: the keys and values
 * of the turn's prompt and of the last f_retained / f_chunk chunks, which the
 * call itself writes in place (the stacked carry of Design, "State rule",
 * Eq. carry: new frames in front, the immutable prompt tail behind, extent
 * capped at L = f_retained + f_prompt; the attended extents are f_prompt,
 * f_prompt + f_chunk, ..., L, Eq. catalog).  The whole call for f_call frames
 * -- n_steps x (input projection, depth x 5 kernels, output projection,
 * guided Euler update) -- is one HIP graph replay (Design, "Granularity and
 * capture placement", Eq. granularity: binding at the chunk clock divides
 * host launches by n_steps).
 *
 * Shapes fixed by the kernels: head width dim / heads = 64 and dim <= 512;
 * mlp a multiple of 32; n_mel a multiple of 8, <= 1024; t_dim even, <= 1024.
 *
 * Conventions are those of dc.h: functions return a dc_status (0 on
 * success); dc_flow_last_error() explains the last failure; a state is not
 * thread-safe; the state owns one device arena whose addresses are fixed
 * until dc_flow_free.  All tensor arguments are device pointers in
 * row-major float32 unless DC_HOST_PTRS is set in flags (then host pointers,
 * and every call is synchronous).
 */
#ifndef DC_FLOW_H
#define DC_FLOW_H

#include <stddef.h>
#include <stdint.h>

#include "dc.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DC_FLOW_ABI_VERSION 1

typedef struct dc_flow_cfg {
    int32_t abi_version;                 /* DC_FLOW_ABI_VERSION                                   */
    int32_t n_mel, dim, heads, depth;    /* estimator: mel bins, width, heads (dim/heads = 64),   */
    int32_t mlp, t_dim;                  /*   blocks, MLP width, sinusoidal time-embedding width  */
    int32_t n_steps;                     /* Euler solver steps per call                           */
    int32_t f_prompt;                    /* largest prompt, frames                                */
    int32_t f_retained;                  /* history frames kept in the carry (multiple of f_chunk)*/
    int32_t f_chunk;                     /* frames a full call retains (its advance)              */
    int32_t f_call;                      /* largest call: f_chunk plus the lookahead              */
    int32_t batch;                       /* independent streams decoded together                  */
    int32_t dtype;                       /* DC_F32 or DC_BF16 (bf16 operands, fp32 accumulation)  */
    uint32_t flags;                      /* DC_HOST_PTRS, DC_NO_GRAPH                             */
    float cfg_rate;                      /* guidance weight w                                     */
    float temperature;                   /* scale of the initial noise                            */
    uint64_t rng_seed;                   /* first key word of the noise generator                 */
    void* hip_stream;                    /* hipStream_t to run on; NULL = a stream of the state's own */
} dc_flow_cfg;

typedef struct dc_flow_stats {
    int64_t calls;            /* dc_flow_decode_chunk calls that launched work                  */
    int64_t replays;          /* calls served by the captured f_call-frame graph                */
    int64_t direct;           /* calls launched kernel by kernel (other n, or DC_NO_GRAPH)       */
    int64_t prompts;          /* dc_flow_prompt calls                                            */
    int64_t rejected;         /* calls refused by argument checks                               */
    int64_t weight_bytes;     /* device bytes of weights and per-step constants                 */
    int64_t carry_bytes;      /* device bytes of the stacked carry (all streams)                */
    int64_t carry_live_bytes; /* bytes of the carry's declared live extent L (all streams)      */
    int64_t arena_bytes;      /* total device bytes of the state                                */
    int32_t kernels_per_call; /* kernel launches of one f_call-frame call                       */
    int32_t graph_nodes;      /* nodes of the captured graph (0 without one)                    */
    double capture_ms;        /* dc_flow_init wall time: upload, constants, warm-up, capture     */
} dc_flow_stats;

/* Device time of one kernel role in one call (dc_flow_profile). */
typedef struct dc_flow_kernel_stat {
    char name[48];            /* role: "assemble", "gemm:in", "gemm:qkv", "attn", "gemm:o",
                                 "gemm:fc1", "gemm:fc2", "gemm:out", "euler"                           */
    int32_t launches;         /* launches of this role per call                                      */
    int32_t mfma;             /* 1: the role is a matrix-core contraction                            */
    double us;                /* device time per call, summed over its launches (HIP events)        */
    double flops;             /* algorithmic floating-point operations per call                      */
    double bytes;             /* algorithmic HBM bytes per call: operands read once, results written */
} dc_flow_kernel_stat;

typedef struct dc_flow_state dc_flow_state;

/* Number of float32 values the weight blob of cfg must hold (0 for NULL).  The
 * blob holds, back to back in PyTorch Linear layouts [out][in]: the time MLP
 * (t.W1 [dim][t_dim], t.b1, t.W2 [dim][dim], t.b2), the input projection
 * (in.W [dim][4 n_mel], in.b), per block (ada.W [6 dim][dim], ada.b,
 * qkv.W [3 dim][dim], qkv.b, o.W [dim][dim], o.b, fc1.W [mlp][dim], fc1.b,
 * fc2.W [dim][mlp], fc2.b) and the final layer (ada.W [2 dim][dim], ada.b,
 * out.W [n_mel][dim], out.b). */
int64_t dc_flow_blob_floats(const dc_flow_cfg* cfg);

/* Create a state: validate cfg, upload the weights (host float32 blob of
 * blob_bytes bytes; rounded to bfloat16 for a DC_BF16 state's per-step Linear
 * layers), compute the per-step time modulations on the device, zero the
 * carry, and capture the f_call-frame call as one graph.  No stream has a
 * turn yet.  Errors: DC_EINVAL (bad cfg or blob size), DC_EVERSION,
 * DC_ENOMEM, DC_EDEVICE. */
dc_status dc_flow_init(const void* weights_blob, size_t blob_bytes, const dc_flow_cfg* cfg, dc_flow_state** out);

/* Start a turn of stream b: the prompt pass over `frames` frames (1 <=
 * frames <= f_prompt; mu and cond [frames][n_mel], spk [n_mel]) writes the
 * prompt's keys and values of every solver step, block and guidance branch
 * in place as the stream's whole carry (the turn transition of Design,
 * "State rule": base state written into existing storage), and restarts the
 * stream's frame position and history.  Other streams are untouched.  Errors:
 * DC_EINVAL (NULL pointer, b or frames out of range), DC_ESTATE, DC_EDEVICE. */
dc_status dc_flow_prompt(dc_flow_state* s, int32_t b, const float* mu, const float* cond, const float* spk,
                         int32_t frames);

/* One chunk call for every stream: mu [batch][n][n_mel] are the features of
 * frames [p_b, p_b + n) of each stream (p_b = the stream's position), mel_out
 * [batch][n][n_mel] receives the solved mel frames.  1 <= n <= f_call; every
 * stream must have a turn.  When n >= f_chunk the first f_chunk frames of
 * each stream enter its carry and its position advances by f_chunk (the rest
 * are the lookahead, presented again by the next call); a call of fewer
 * frames is a flush that changes no state.  n == f_call replays the captured
 * graph.  Errors: DC_EINVAL, DC_ERANGE (n out of range), DC_ESTATE (a stream
 * without a turn, or a poisoned state), DC_EDEVICE. */
dc_status dc_flow_decode_chunk(dc_flow_state* s, const float* mu, int32_t n, float* mel_out);

/* Wait for the state's stream. */
dc_status dc_flow_sync(dc_flow_state* s);

/* The carry of stream b for (solver step, block, branch 0 = conditional /
 * 1 = unconditional, kv 0 = keys / 1 = values) in Eq. carry's logical order
 * (newest retained chunk first, the prompt last), widened to float32 into the
 * host buffer host_out [frames][dim]; *frames receives the extent.  Pass
 * host_out = NULL to query the extent.  For audits against the definition
 * (the shadow auditor of Design, "Verification"); synchronous.  Errors:
 * DC_EINVAL, DC_EDEVICE. */
dc_status dc_flow_carry_read(dc_flow_state* s, int32_t b, int32_t step, int32_t layer, int32_t branch, int32_t kv,
                             float* host_out, int32_t* frames);

dc_status dc_flow_get_stats(const dc_flow_state* s, dc_flow_stats* out);

/* Time an f_call-frame call launch by launch, `reps` times (mean per call),
 * with HIP events on the state's stream, grouped by kernel role into out[0 ..
 * *count) (at most max entries; out = NULL queries the count).  The streams'
 * state does not advance and no retained frame changes: the call writes only
 * the slot that the next call overwrites.  Every stream needs a turn.  For
 * measurement; synchronous.  Errors: DC_EINVAL, DC_ESTATE, DC_EDEVICE. */
dc_status dc_flow_profile(dc_flow_state* s, int32_t reps, dc_flow_kernel_stat* out, int32_t max, int32_t* count);

/* Text of the last error of s (of the last failed dc_flow_init when s is NULL). */
const char* dc_flow_last_error(const dc_flow_state* s);

/* Release the state and its device memory.  NULL is a no-op. */
void dc_flow_free(dc_flow_state* s);

#ifdef __cplusplus
}
#endif

#endif
