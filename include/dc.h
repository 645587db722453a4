/*
 * dc.h — C ABI of the MI355X streaming Token2Wav decode step.
 *
 * One call to dc_decode_chunk turns a chunk of n speech tokens per stream into
 * fp32 PCM: token embedding repeated to the frame clock, a causal Conv1d
 * pre-stack, ConvTranspose1d upsampling stages each followed by a
 * multi-receptive-field residual block, a head conv to log-magnitude and phase,
 * and an inverse STFT with overlap-add.  Every causal layer reads its left
 * context from a ring buffer kept at a fixed device address (the carry of the
 * paper's state rule: Design, "State rule: demand sizing and the carry",
 * Eq. carry), written in place by the kernel that produces it; the whole step
 * for the declared chunk shape is replayed as one HIP graph (the compute rule:
 * Design, "Compute rule: exact-shape replay", clauses (i)-(ii), Eq. granularity).
 *
 * Correctness contract (Design, Definition 2, strict trace equivalence): for
 * every stream, decoding a token sequence chunk by chunk yields bit-for-bit the
 * PCM of decoding the concatenation in one call, and graph replay yields
 * bit-for-bit the PCM of direct launches.  This holds within one state and
 * across states that share the architecture, dtype and batch class: with the
 * automatic tile choice (tile_variant 0) the reduction order of every output
 * sample depends on the layer, the dtype and whether batch < 8 (the streaming
 * class: K split in four partitions) or batch >= 8 (the batched class: one
 * partition, bf16 resblock pairs fused), never on chunk_tokens, max_tokens,
 * the call's n or the stream's index in the batch.  A fresh state whose
 * chunk_tokens covers a whole utterance therefore decodes it to the bits of a
 * chunked decode on a state of the same class.  Across classes the PCM
 * agrees within the rounding tolerance of the dtype, not bit for bit.
 *
 * Conventions for every function:
 *   - the return value is a dc_status (0 on success, negative on error); no
 *     exception or abort crosses the ABI; dc_last_error() explains the last one;
 *   - a dc_state is not thread-safe; distinct states are independent;
 *   - the state owns all device memory it allocates (one arena at dc_init); its
 *     addresses are fixed until dc_free.
 */
#ifndef DC_H
#define DC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DC_ABI_VERSION 3
#define DC_MAX_STAGES 4
#define DC_MAX_RB 4
#define DC_MAX_DIL 4

typedef enum {
    DC_OK = 0,
    DC_EINVAL = -1,   /* bad argument or configuration; nothing launched, state unchanged */
    DC_ERANGE = -2,   /* token id outside [0, vocab) or n > max_tokens                      */
    DC_ENOMEM = -3,   /* device allocation failed at dc_init                                 */
    DC_EDEVICE = -4,  /* a HIP call failed; the state is poisoned until dc_reset             */
    DC_ESTATE = -5,   /* the state is poisoned (earlier device or id error); call dc_reset   */
    DC_EVERSION = -6  /* cfg->abi_version != DC_ABI_VERSION                                  */
} dc_status;

typedef enum { DC_F32 = 0, DC_BF16 = 1 } dc_dtype;

enum {
    DC_HOST_PTRS = 1u << 0, /* tokens/audio are host pointers; each call is synchronous          */
    DC_NO_GRAPH = 1u << 1,  /* never capture or replay a graph; always launch kernels directly   */
    DC_NO_FUSE = 1u << 2,   /* run every resblock conv as its own launch (no fused pairs)        */
    DC_FLUSH_CATALOG = 1u << 3, /* also capture one graph per partial-chunk size n in [1, chunk_tokens)
                                  (Design, "Scope: catalog width": a flush at a turn boundary adds
                                  at most one class per admissible extent below the chunk); not
                                  with DC_NO_GRAPH                                                 */
    DC_NO_RING = 1u << 4    /* bf16 convs never stage weights through the LDS ring (ablation);
                               the PCM is bit-identical either way                                */
};

/*
 * Decoder architecture and serving shape.  The architecture fields describe
 * the weight blob (see dc_init); the serving fields size the state.
 * Constraints checked by dc_init (DC_EINVAL otherwise): 1 <= n_stages <= 4,
 * channels multiples of 8, channels[0] == embed, 1 <= n_rb <= 4,
 * 1 <= n_dil <= 4, odd or even kernels >= 1, n_fft == 16 and hop == 4,
 * batch >= 1, 1 <= chunk_tokens <= max_tokens.
 */
typedef struct dc_cfg {
    int32_t abi_version;                 /* DC_ABI_VERSION                                        */
    int32_t vocab, embed;                /* token vocabulary, embedding width                     */
    int32_t frames_per_token;            /* embedding repeat to the frame clock                  */
    int32_t n_pre, pre_kernel;           /* causal Conv1d pre-stack (dilation 1)                  */
    int32_t n_stages;                    /* upsampling stages                                     */
    int32_t up_rate[DC_MAX_STAGES];      /* stride u of each ConvTranspose1d (kernel 2u)          */
    int32_t channels[DC_MAX_STAGES + 1]; /* channels[0] pre-stack width, channels[s+1] stage s    */
    int32_t n_rb, rb_kernel[DC_MAX_RB];  /* resblock kernel sizes (one branch each)               */
    int32_t n_dil, dil[DC_MAX_DIL];      /* dilations of every branch                             */
    int32_t head_kernel, n_fft, hop;     /* head conv width, iSTFT size and hop                   */
    float lrelu_slope;                   /* LeakyReLU negative slope                              */
    int32_t dtype;                       /* dc_dtype: arithmetic of the conv operands             */
    int32_t batch;                       /* B independent streams sharing the weights             */
    int32_t chunk_tokens;                /* the chunk shape captured as a graph                   */
    int32_t max_tokens;                  /* largest n accepted by dc_decode_chunk                 */
    uint32_t flags;                      /* DC_HOST_PTRS | DC_NO_GRAPH | DC_NO_FUSE | DC_FLUSH_CATALOG |
                                            DC_NO_RING */
    int32_t tile_variant;                /* 0: automatic; v > 0 forces tile shape v-1, and with it
                                            its K partitions and channel block, everywhere it fits
                                            (shapes that share those two give identical results) */
    /* Harmonic-plus-noise excitation source (the vocoder's stochastic input;
     * n_harmonics == 0: none, and the fields below are ignored).  Per frame of
     * the pre-stack clock the caller gives f0 (Hz); the source sums the
     * fundamental and n_harmonics overtones (amplitude sine_amp, voiced where
     * f0 > voiced_threshold) and Gaussian noise (noise_std when voiced,
     * sine_amp / 3 when not) drawn from Philox4x64-10 keyed by (rng_seed,
     * stream index) with the sample index since the stream's start as
     * counter, merges them with a learned linear layer and tanh, and adds it
     * to the last stage through a Conv1d with kernel = stride = hop after the
     * stage's ConvTranspose1d. */
    int32_t n_harmonics;                 /* overtones besides the fundamental, 0..31              */
    float sine_amp, noise_std;           /* sinusoid amplitude, voiced noise standard deviation   */
    float voiced_threshold;              /* Hz                                                    */
    float sample_rate;                   /* Hz of the output samples                              */
    uint64_t rng_seed;                   /* key of the source's counter-based generator           */
    void* hip_stream;                    /* hipStream_t all work is ordered on; NULL: own stream  */
} dc_cfg;

typedef struct dc_stats {
    int64_t calls;            /* dc_decode_chunk calls that launched work                       */
    int64_t replays;          /* ... of which replayed a captured graph (chunk or flush class)  */
    int64_t direct_shape;     /* direct launches because no class was captured for n            */
    int64_t direct_nograph;   /* direct launches because no graph exists (DC_NO_GRAPH)          */
    int64_t staged_tokens;    /* token copies into the fixed token buffer (caller not aliased)  */
    int64_t staged_audio;     /* PCM copies out of the fixed audio buffer (caller not aliased)  */
    int64_t rejected;         /* calls refused before any launch                                */
    int64_t clock_tokens;     /* tokens decoded per stream since the last dc_reset              */
    int64_t arena_bytes;      /* the one device allocation                                      */
    int64_t weight_bytes;     /* packed weights and device-resident constants                   */
    int64_t carry_bytes;      /* left-context part of every ring (the state kept across chunks) */
    int64_t ring_bytes;       /* all ring buffers (carry plus the frames of one call)           */
    int32_t kernels_per_step; /* kernel launches of one chunk step                              */
    int32_t graph_nodes;      /* nodes of the captured graph (0 if none)                        */
    double capture_ms;        /* wall time of warm-up, capture and instantiation at dc_init     */
    int64_t replays_flush;    /* replays of a partial-chunk class (DC_FLUSH_CATALOG)            */
    int32_t graph_classes;    /* captured shape classes: 0, 1 or chunk_tokens                   */
    int32_t reserved;
    int64_t staged_f0;        /* f0 copies into the fixed f0 buffer (caller not aliased)        */
    int64_t direct_static;    /* direct launches of dc_decode_chunk_f0_static                   */
} dc_stats;

typedef struct dc_state dc_state;

/*
 * Create a decoder.  weights_blob: host pointer to blob_bytes of little-endian
 * float32, the tensors back to back in this order and PyTorch layouts:
 *   emb [vocab][embed];
 *   per pre layer: W [C0][C0][pre_kernel], b [C0];
 *   per stage s: ConvTranspose1d W [C_s][C_{s+1}][2*u_s], b [C_{s+1}], then per
 *     resblock kernel k_j, per dilation d: W1 [C][C][k_j], b1 [C], W2 [C][C][k_j], b2 [C];
 *   head: W [2*(n_fft/2+1)][C_last][head_kernel], b [2*(n_fft/2+1)];
 *   with a harmonic source (n_harmonics > 0): merge W [n_harmonics+1],
 *     merge b [1], down W [C_last][1][hop], down b [C_last].
 * The blob is copied (rounded to bfloat16, nearest-even, when dtype is
 * DC_BF16; the head stays fp32 arithmetic on those rounded values) and may be
 * freed on return.  A DC_BF16 state stores the stages' residual stream (the
 * "s<s>.y", "s<s>.rb<j>.z<i>" and "s<s>.x" intermediates) as IEEE binary16:
 * activations of order one keep 11 significant bits; magnitudes beyond
 * 65504 do not fit (a DC_F32 state has no such limit): a value that would
 * round to infinity (|v| >= 65520), or a NaN, raises the device flag, which
 * the next dc_sync reports as DC_ERANGE (the state is poisoned until dc_reset).  On success *out owns the state, reset to the start of
 * every stream, with the chunk graph captured unless DC_NO_GRAPH.
 * Errors: DC_EVERSION, DC_EINVAL (cfg or blob size), DC_ENOMEM, DC_EDEVICE;
 * *out is NULL then.
 */
dc_status dc_init(const void* weights_blob, size_t blob_bytes, const dc_cfg* cfg, dc_state** out);

/*
 * Decode the next n tokens of every stream.
 *   tokens:    int32 [batch][n], row-major.
 *   audio_out: float32 [batch][n * dc_samples_per_token(cfg)], row-major; the
 *              samples continue each stream where the previous call ended.
 * Pointers are device pointers ordered on the state's stream (asynchronous)
 * unless the state was created with DC_HOST_PTRS (synchronous, host memory).
 * Passing dc_token_buffer(s) / dc_audio_buffer(s) aliases the fixed buffers and
 * avoids the staging copy of that side.
 * Admission (Design, compute rule clauses (i)-(ii), fail-closed): n ==
 * chunk_tokens replays the captured graph; with DC_FLUSH_CATALOG so does
 * 0 < n < chunk_tokens (its own class, counted in replays and replays_flush);
 * any other 0 < n <= max_tokens runs the same kernels directly (bit-identical
 * output, counted as direct_shape).
 * n <= 0 or NULL pointers: DC_EINVAL; n > max_tokens: DC_ERANGE; both leave
 * the state unchanged.  Token ids outside [0, vocab): with DC_HOST_PTRS,
 * DC_ERANGE before any launch, state unchanged; with device pointers the
 * embedding kernel raises a device flag, and this call (host mode) or the
 * next dc_sync returns DC_ERANGE and poisons the state until dc_reset.
 */
dc_status dc_decode_chunk(dc_state* s, const int32_t* tokens, int32_t n, float* audio_out);

/*
 * dc_decode_chunk for a decoder with a harmonic source (n_harmonics > 0;
 * dc_decode_chunk refuses such a state with DC_EINVAL, and this call refuses
 * a state without one).  f0: float32 [batch][n * frames_per_token], Hz per
 * frame of the pre-stack clock, in the same pointer space as tokens (passing
 * dc_f0_buffer(s) aliases the fixed buffer).  The source's draws and phases
 * depend only on each stream's samples since its start, so a chunked decode
 * equals an offline one bit for bit, and a graph replay equals a direct
 * launch (Design, clause (iii): the device generator advances along a
 * declared clock).  Errors as dc_decode_chunk, plus DC_EINVAL for a NULL f0.
 */
dc_status dc_decode_chunk_f0(dc_state* s, const int32_t* tokens, const float* f0, int32_t n, float* audio_out);

/*
 * dc_decode_chunk_f0 for callers that cannot allocate device memory or must
 * not have the library do so on their behalf (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the call's one
 * scratch buffer -- the harmonic source's table of phases at the start of
 * every f0 frame, batch * n * frames_per_token * (n_harmonics + 1) doubles --
 * lives in a file-scope device array of the library (4 MiB, one copy per
 * device for the life of the process, its address resolved at the dc_init of
 * the first decoder with a source on that device) instead of the state's
 * arena.  The call allocates nothing, captures nothing and always launches
 * the step's kernels directly (counted as direct_static); tokens, f0 and
 * audio_out are as for dc_decode_chunk_f0, and the PCM is bit-identical to
 * it.  The array keeps the last call's contents, which every call overwrites
 * before reading; all calls on one device share it, so calls that overlap in
 * time on one device (states on different streams) race and must be
 * serialised by the caller.  Errors: as dc_decode_chunk_f0, plus DC_ERANGE
 * (nothing launched, state unchanged) when the phase table would exceed
 * 4 MiB, and DC_EINVAL for a decoder without a harmonic source.
 */
dc_status dc_decode_chunk_f0_static(dc_state* s, const int32_t* tokens, const float* f0, int32_t n,
                                    float* audio_out);

/* Return every stream to its start: zero every ring in place (addresses are
 * unchanged) and set the clock to 0.  Clears a poisoned state.  This is the
 * state rule's reset, which writes the base state into the contract-owned
 * carry in place rather than reallocating it (Design, "State rule: demand
 * sizing and the carry"; the representation invariant that every replay sees
 * the same addresses). */
dc_status dc_reset(dc_state* s);

/* Return stream b (0 <= b < batch) to its start in place; other streams keep
 * their carry (the state rule's in-place reset applied to one session's slice
 * of the carry, as a turn boundary of one session of a multi-session binding
 * needs).  DC_EINVAL for a bad b. */
dc_status dc_reset_stream(dc_state* s, int32_t b);

/* Wait for all work of the state; report DC_ERANGE for a bad token id seen on
 * the device or, in a DC_BF16 state, a residual-stream value beyond the
 * binary16 range, DC_EDEVICE for a HIP error (all poison the state; the
 * message names which).  A failure
 * found here is the device side of the fail-closed admission: the call that
 * raised it produced no trusted output (Design, "Granularity and capture
 * placement", local fail-closed admission). */
dc_status dc_sync(dc_state* s);

/* frames_per_token * prod(up_rate) * hop for cfg (0 for a NULL cfg or one
 * that dc_init would reject as invalid). */
int64_t dc_samples_per_token(const dc_cfg* cfg);

/* Number of float32 values the weight blob of cfg must hold (0 for a NULL or
 * invalid cfg). */
int64_t dc_blob_floats(const dc_cfg* cfg);

/* The fixed device buffers that dc_decode_chunk stages through:
 * int32 [batch][max_tokens] and float32 [batch][max_tokens * samples_per_token]
 * (read as [batch][n] and [batch][n * spt] for a call with n tokens).  A
 * caller that writes its tokens here and reads its PCM from here is aliased
 * with the contract's own inputs and outputs, so no staging copy is made on
 * that side (Design, clause (ii) address stability: contract-owned inputs are
 * aliased and skip per-call staging; Proposition 2, mutual enabling, and Eq.
 * enabling: an aliased input needs no class-specific staging storage).  Owned by the state; valid until
 * dc_free. */
int32_t* dc_token_buffer(dc_state* s);
float* dc_audio_buffer(dc_state* s);

/* The fixed device f0 buffer of a decoder with a harmonic source: float32
 * [batch][max_tokens * frames_per_token] (read as [batch][n * frames_per_token]);
 * NULL without a source. */
float* dc_f0_buffer(dc_state* s);

/*
 * Carry snapshots: time-multiplexing many sessions over the streams of one
 * state, and checkpoint/resume (the paper's O(1) carry per session: Design,
 * state rule, Eq. carry; multi-session bindings).  A snapshot of stream b
 * holds what its next call reads from the past -- every ring's left context
 * (the ctx frames before the stream's position), the harmonic source's phases
 * -- plus the stream's position (tokens since its start) and its source
 * generator key.  dc_carry_import places a snapshot into stream b of a state
 * with the same architecture, dtype, source and ring layout (a fused state,
 * bf16 with batch >= 8, lays its rings out differently from an unfused one):
 * the frames go to the slots of that state's own clock and the stream's start
 * is placed `position` tokens back, so the stream continues there bit for bit
 * as if it had never left.  Other streams are untouched.  Both calls are
 * synchronous and take a host buffer of exactly dc_carry_bytes(s) bytes.
 * Errors: DC_EINVAL (bad b, NULL or wrong-size buffer, a snapshot of another
 * layout), DC_ESTATE (poisoned state), DC_EDEVICE.
 */
int64_t dc_carry_bytes(const dc_state* s);
dc_status dc_carry_export(dc_state* s, int32_t b, void* host_out, size_t bytes);
dc_status dc_carry_import(dc_state* s, int32_t b, const void* host_in, size_t bytes);

/* Copy the counters into *out. */
dc_status dc_get_stats(const dc_state* s, dc_stats* out);

/*
 * Inspection of the carried state and intermediates (tests, shadow checks).
 * dc_tap_find returns the index of a named intermediate ("embed", "pre<l>",
 * "s<s>.y", "s<s>.rb<j>.h<i>" (stored as LeakyReLU of h), "s<s>.rb<j>.z<i>",
 * "s<s>.x", "head", and with a harmonic source "src": its samples as frames
 * of the last stage's clock, hop samples each), or -1.  dc_tap_read copies, for stream b, the frames
 * with absolute index [frame0, frame0 + nframes) of that ring into host
 * memory as float32 [nframes][C]; *channels receives C.  Only frames still held
 * by the ring (the last call's frames and the carried left context) are
 * readable; others give DC_ERANGE.  Where a resblock pair runs fused (bf16,
 * batch >= 8, 64 or 128 channels, unless DC_NO_FUSE), its h stays on chip and
 * the "h" intermediate holds no frames (DC_ERANGE).  Synchronous.
 */
int32_t dc_tap_find(const dc_state* s, const char* name);
dc_status dc_tap_read(dc_state* s, int32_t tap, int32_t b, int64_t frame0, int32_t nframes,
                      float* host_out, int32_t* channels);

/*
 * Measurement (roofline reporting).  A chunk step is a fixed sequence of
 * kernel launches ("layers": embed, each conv / transposed conv -- the
 * convs at one position of the parallel resblock branches share a launch,
 * and a fused resblock pair is one launch --,
 * head, the iSTFT tail, which also advances the clock).  dc_layer_info
 * describes launch i at
 * n = chunk_tokens: its kernel (the demangled name a profiler shows), the
 * GEMM shape of a conv (rows = batch * frames, cols, depth = taps * input
 * channels, summed over the launch's convs), its algorithmic FLOPs (2 *
 * multiply-adds of the convolutions) and its algorithmic HBM bytes (weights
 * once, operand frames including left context, residual / branch inputs,
 * output frames).  dc_time_layers launches
 * every layer reps times in isolation on the state's stream, bracketed by HIP
 * events, and writes the mean microseconds per launch into us_per_launch
 * [dc_layer_count].  Re-running a layer rewrites only ring slots of frames the
 * next call overwrites anyway, and a re-run iSTFT tail leaves the clock where
 * it is, so the stream state is unaffected.  Synchronous.
 */
typedef struct dc_layer_info {
    char name[48];
    char kernel[80];
    int64_t rows, cols, depth;
    double flops;
    double bytes;
} dc_layer_info;

int32_t dc_layer_count(const dc_state* s);
dc_status dc_layer_info_get(const dc_state* s, int32_t i, dc_layer_info* out);
dc_status dc_time_layers(dc_state* s, int32_t reps, double* us_per_launch);

/* Bounds checks of the checked build (libdc_debug.so, the same sources built
 * with DC_DEBUG): every ring access of the kernels (operand, output,
 * residual, branch-mean, source, z, head, iSTFT and embedding rings) and the
 * row range of every staged operand tile is checked; a failed check sets its
 * bit and the access is redirected to element 0 of its buffer.  Returns the
 * OR of the bits set on the current device since the last clear (0: none),
 * clearing them if clear != 0, after waiting for the device; -1 from the
 * release build (checks compiled out), -2 on a HIP error.  Bits: 1 operand
 * ring, 2 operand tile rows, 4 conv output/residual/mean/source rings, 8 fused
 * pair z ring, 16 fused pair output/mean rings, 32 iSTFT tail, 64 embedding. */
int32_t dc_debug_checks(int32_t clear);

/* Human-readable reason for the last error on s (or on dc_init when s is NULL). */
const char* dc_last_error(const dc_state* s);

/* Release the state and all its device memory (NULL is a no-op). */
void dc_free(dc_state* s);

#ifdef __cplusplus
}
#endif

#endif /* DC_H */
