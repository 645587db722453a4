// Host runtime of the streaming Token2Wav decode step: configuration checks,
// weight packing, the one device arena, the carried ring buffers, the device
// clock, fail-closed admission, HIP-graph capture and replay, counters.
//
// State rule (Design, "State rule: demand sizing and the carry", Eq. carry):
// every intermediate a causal layer reads is a ring of ctx + F_max frames per
// stream at a fixed address, where ctx is exactly the left context its
// consumers read ((k-1)*d for a conv, 1 frame for a transposed conv, n_fft/hop
// - 1 windowed frames for the overlap-add) and F_max the frames of the largest
// call.  The producing kernel writes a call's frames at slots tau mod R, so
// the left context of the next call is already in place: no staging copy, no
// pointer change, and a reset zeroes the rings where they are.
//
// Compute rule (Design, "Compute rule: exact-shape replay", Eq. granularity):
// the whole chunk step for n == chunk_tokens is captured once as one HIP
// graph and replayed; kernels take the time offset of a call from a device
// clock that the last node advances, so the frozen kernel arguments stay
// valid.  Any other admissible n launches the same kernels directly.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <limits>
#include <mutex>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/dc.h"
#include "dc_internal.h"

using namespace dc;

namespace {

struct ConvOp {
    std::string name;
    int in = -1, out = -1, res = -1;
    int mean[3] = {-1, -1, -1};
    int n_mean = 0;
    int Ci = 0, N = 0, out_C = 0, k = 1, d = 1, u = 1;
    int in_act = 0, out_act = 0;
    bool bf16 = false;   // operand type
    bool split = false;  // bf16 operand as a hi + lo pair
    bool transposed = false;
    size_t w_off = 0, b_off = 0, w_bytes = 0;
    size_t blob_w = 0, blob_b = 0;  // float offsets into the blob
    int CB = 0, n_cb = 0, NB16 = 0;
    int variant = 0;
    int level_in = 0;
    int stage = -1, branch = -1, dil_i = -1, half = 0;   // resblock position (-1: not a resblock conv)
    int partner = -1;    // fused pair: the other conv of the pair (h stays on chip)
    int src_ring = -1;   // the last stage's ConvTranspose1d with a harmonic source: its samples
};

// One kernel launch of a chunk step.
enum LaunchKind { L_EMBED, L_CONV, L_PAIR, L_ISTFT, L_PHASE, L_SOURCE };
struct Launch {
    LaunchKind kind;
    std::vector<int> convs;   // members of a conv launch (same tile shape; parallel branches);
                              // of a pair launch, each member's first conv
    std::string name;
    int pair_variant = 0;     // L_PAIR: fused-pair shape
};

thread_local std::string g_init_error;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

uint16_t host_f2bf(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0x007fffffu) ? 0x40u : 0u));
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

float host_bf2f(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// IEEE binary16 bits -> float.
float host_h2f(uint16_t h)
{
    const int e = (h >> 10) & 31, m = h & 1023;
    const float sgn = (h & 0x8000) ? -1.f : 1.f;
    if (e == 31) return m ? std::numeric_limits<float>::quiet_NaN() : sgn * std::numeric_limits<float>::infinity();
    return sgn * std::ldexp((float)(e ? (1024 + m) : m), (e ? e : 1) - 25);
}

float round_param(float x, bool bf16) { return bf16 ? host_bf2f(host_f2bf(x)) : x; }

}  // namespace

struct dc_state {
    dc_cfg cfg{};
    hipStream_t stream = nullptr;
    bool own_stream = false;
    // harmonic source: its two launches run on a side stream, forked at the
    // step's start and joined before the launch that adds the source
    hipStream_t side = nullptr;
    hipEvent_t fork_ev = nullptr, join_ev = nullptr;
    int src_join = -1;          // index of the launch that reads the source ring
    char* arena = nullptr;
    size_t arena_bytes = 0;
    std::vector<Ring> rings;
    std::vector<std::string> ring_names;
    std::vector<int> ring_ctx;
    std::vector<bool> ring_onchip;   // h of a fused pair: never materialised (R = 0)
    std::vector<ConvOp> convs;
    std::vector<Launch> launches;
    int ring_E = -1, ring_S = -1, ring_G = -1, ring_src = -1;
    int levels = 0;
    int64_t fpt[DC_MAX_STAGES + 2] = {};
    int64_t spt = 0;
    size_t emb_off = 0, table_off = 0, tok_off = 0, audio_off = 0, clock_off = 0, start_off = 0, err_off = 0;
    size_t arrivals_off = 0;
    size_t keys_off = 0;
    // harmonic source: merge weights and bias, down-conv weights and bias,
    // the f0 buffer, the carried phases and the per-call phase table
    size_t src_w_off = 0, src_down_off = 0, f0_off = 0, phase_off = 0, ptab_off = 0;
    float* f0 = nullptr;
    size_t ring_begin = 0, ring_end = 0;
    int32_t* tok = nullptr;
    float* audio = nullptr;
    int64_t* clock = nullptr;
    int64_t* start = nullptr;   // [B] tokens decoded when each stream last started
    uint64_t* keys = nullptr;   // [B] each stream's source-generator key
    int* err = nullptr;
    unsigned* arrivals = nullptr;   // blocks of the running iSTFT launch that are done (zero between calls)
    void* emb = nullptr;
    float* table = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    // DC_FLUSH_CATALOG: one class per partial-chunk size n (index n, 1 <= n < chunk_tokens)
    std::vector<hipGraph_t> flush_graph;
    std::vector<hipGraphExec_t> flush_exec;
    dc_stats st{};
    int device = 0;             // the device current at dc_init (the arena's)
    double* static_ptab = nullptr;   // that device's static scratch (harmonic source only)
    int64_t clock_host = 0;
    bool poisoned = false;
    std::string msg;
};

// ------------------------------------------------------------------ helpers

static dc_status fail(dc_state* s, dc_status code, const std::string& why)
{
    if (s) s->msg = why;
    else g_init_error = why;
    return code;
}

static dc_status device_fail(dc_state* s, hipError_t e, const char* where)
{
    s->poisoned = true;
    return fail(s, DC_EDEVICE, std::string(where) + ": " + hipGetErrorString(e));
}

static int64_t samples_per_token(const dc_cfg* c)
{
    int64_t u = 1;
    for (int i = 0; i < c->n_stages; i++) u *= c->up_rate[i];
    return (int64_t)c->frames_per_token * u * c->hop;
}

static int64_t blob_floats(const dc_cfg* c)
{
    int64_t n = (int64_t)c->vocab * c->embed;
    int64_t c0 = c->channels[0];
    n += (int64_t)c->n_pre * (c0 * c0 * c->pre_kernel + c0);
    for (int s = 0; s < c->n_stages; s++) {
        int64_t ci = c->channels[s], co = c->channels[s + 1];
        n += ci * co * 2 * c->up_rate[s] + co;
        for (int j = 0; j < c->n_rb; j++) n += (int64_t)c->n_dil * 2 * (co * co * c->rb_kernel[j] + co);
    }
    int64_t hc = 2 * (c->n_fft / 2 + 1);
    n += hc * c->channels[c->n_stages] * c->head_kernel + hc;
    if (c->n_harmonics > 0) n += (c->n_harmonics + 1) + 1 + (int64_t)c->channels[c->n_stages] * c->hop + c->channels[c->n_stages];
    return n;
}

static constexpr int kMaxSinusoidsHost = 32;   // the source kernel's bound on n_harmonics + 1

static std::string validate(const dc_cfg* c)
{
    if (c->vocab <= 0 || c->embed <= 0) return "vocab and embed must be positive";
    if (c->frames_per_token < 1 || c->frames_per_token > 64) return "frames_per_token must be in [1, 64]";
    if (c->n_pre < 0 || c->n_pre > 64 || c->pre_kernel < 1 || c->pre_kernel > 64) return "bad pre-stack";
    if (c->n_stages < 1 || c->n_stages > DC_MAX_STAGES) return "n_stages must be in [1, 4]";
    for (int i = 0; i < c->n_stages; i++)
        if (c->up_rate[i] < 1 || c->up_rate[i] > 64) return "up_rate must be in [1, 64]";
    for (int i = 0; i <= c->n_stages; i++)
        if (c->channels[i] < 8 || c->channels[i] % 8 || c->channels[i] > 4096)
            return "channels must be positive multiples of 8 (<= 4096)";
    if (c->channels[0] != c->embed) return "channels[0] must equal embed";
    if (c->n_rb < 1 || c->n_rb > DC_MAX_RB) return "n_rb must be in [1, 4]";
    for (int i = 0; i < c->n_rb; i++)
        if (c->rb_kernel[i] < 1 || c->rb_kernel[i] > 64) return "rb_kernel must be in [1, 64]";
    if (c->n_dil < 1 || c->n_dil > DC_MAX_DIL) return "n_dil must be in [1, 4]";
    for (int i = 0; i < c->n_dil; i++)
        if (c->dil[i] < 1 || c->dil[i] > 64) return "dil must be in [1, 64]";
    if (c->head_kernel < 1 || c->head_kernel > 64) return "head_kernel must be in [1, 64]";
    if (c->n_fft != 16 || c->hop != 4) return "only n_fft = 16, hop = 4 is supported";
    if (!(c->lrelu_slope >= 0.0f && c->lrelu_slope <= 1.0f)) return "lrelu_slope must be in [0, 1]";
    if (c->dtype != DC_F32 && c->dtype != DC_BF16) return "dtype must be DC_F32 or DC_BF16";
    if (c->batch < 1 || c->batch > 65536) return "batch must be in [1, 65536]";
    if (c->chunk_tokens < 1 || c->max_tokens < c->chunk_tokens) return "need 1 <= chunk_tokens <= max_tokens";
    if ((int64_t)c->max_tokens * samples_per_token(c) > (int64_t)1 << 30) return "max_tokens too large";
    if (c->flags & ~(uint32_t)(DC_HOST_PTRS | DC_NO_GRAPH | DC_NO_FUSE | DC_FLUSH_CATALOG | DC_NO_RING))
        return "unknown flag bits";
    if ((c->flags & DC_FLUSH_CATALOG) && (c->flags & DC_NO_GRAPH)) return "DC_FLUSH_CATALOG needs graphs (not DC_NO_GRAPH)";
    if (c->tile_variant < 0 || c->tile_variant > num_tile_variants()) return "tile_variant out of range";
    if (c->n_harmonics < 0 || c->n_harmonics >= kMaxSinusoidsHost) return "n_harmonics must be in [0, 31]";
    if (c->n_harmonics > 0) {
        if (!(c->sine_amp >= 0.0f && c->sine_amp < 1e6f) || !(c->noise_std >= 0.0f && c->noise_std < 1e6f))
            return "sine_amp and noise_std must be finite and >= 0";
        if (!(c->sample_rate > 0.0f && c->sample_rate < 1e9f)) return "sample_rate must be positive";
        if (!(c->voiced_threshold > -1e30f && c->voiced_threshold < 1e30f)) return "voiced_threshold must be finite";
    }
    return "";
}

// Geometry of the packed weights of one conv for its tile shape: channel
// block CB = K quantum x KCH channels, ceil(Ci / CB) blocks (zero padded).
static void set_blocks(ConvOp& op)
{
    const int kq = op.bf16 ? 32 : 16;
    op.CB = kq * tile_variant(op.variant).KCH;
    op.n_cb = (op.Ci + op.CB - 1) / op.CB;
    op.NB16 = (op.N + 15) / 16;
    op.w_bytes = (size_t)op.n_cb * op.k * (op.CB / kq) * op.NB16 * 64 * 16;
}

// Weight value of column n, input channel ch, tap j (0 outside the layer).
static float weight_at(const ConvOp& op, const float* blob, int n, int ch, int j)
{
    if (n >= op.N || ch >= op.Ci) return 0.0f;
    if (!op.transposed) return blob[op.blob_w + ((size_t)n * op.Ci + ch) * op.k + j];
    // transposed conv [Ci][Co][2u]: column n = r*Co + o; tap 0 reads the
    // previous input frame (kernel index r + u), tap 1 the current one (r).
    const int r = n / op.out_C, o = n % op.out_C;
    return blob[op.blob_w + ((size_t)ch * op.out_C + o) * (2 * op.u) + r + (1 - j) * op.u];
}

// Pack into MFMA fragment order: [cb][tap][chunk][col block][lane][values].
static void pack_weights(const ConvOp& op, const float* blob, bool round_bf16, char* dst)
{
    const int kq = op.bf16 ? 32 : 16;
    const int chunks = op.CB / kq;
    size_t idx = 0;
    for (int cb = 0; cb < op.n_cb; cb++)
        for (int j = 0; j < op.k; j++)
            for (int kc = 0; kc < chunks; kc++)
                for (int nb = 0; nb < op.NB16; nb++)
                    for (int lane = 0; lane < 64; lane++) {
                        const int n = nb * 16 + (lane & 15);
                        if (op.bf16) {
                            uint16_t* o = (uint16_t*)dst + idx * 8;
                            for (int e = 0; e < 8; e++) {
                                const int ch = cb * op.CB + kc * 32 + (lane >> 4) * 8 + e;
                                o[e] = host_f2bf(weight_at(op, blob, n, ch, j));
                            }
                        } else {
                            float* o = (float*)dst + idx * 4;
                            for (int q = 0; q < 4; q++) {
                                const int ch = cb * op.CB + kc * 16 + (lane >> 4) * 4 + q;
                                o[q] = round_param(weight_at(op, blob, n, ch, j), round_bf16);
                            }
                        }
                        idx++;
                    }
}

// The batch class: from this many streams a state runs every conv with one K
// partition (and, for bf16, the resblock pairs fused); below it, 4.
#ifndef DC_BATCHED_MIN
#define DC_BATCHED_MIN 8
#endif

// Unsplit tile shapes in order of preference (ids of the kernel's shape
// table).  Layers that read a residual and write fp32 -- and every layer of
// the 64-channel stage -- move more bytes per FLOP and run best on 64x64
// tiles, whose lower register use keeps more waves (and loads) in flight;
// the others favour 64x128 tiles (four waves per SIMD with the step
// pipeline), then 128x128.
static const int kPreferLarge[] = {11, 14, 12, 13, 9, 10, 15, 16, 28, 8, 6, 7, 19};
static const int kPrefer64[] = {9, 10, 11, 12, 13, 14, 15, 16, 28, 8, 6, 7, 19};

// LDS budget of one block: at most 80 KB of the CU's 160 KB, so two blocks
// stay resident.
static bool variant_fits(const ConvOp& op, int v)
{
    ConvParams p{};
    p.k = op.k;
    p.d = op.d;
    p.split = op.split;
    const TileShape t = tile_variant(v);
    if (t.W && !op.bf16) return false;   // the LDS weight ring exists for bf16 operands only
    const int npad = (op.N + 15) / 16 * 16;
    return conv_lds_bytes(v, op.bf16, p) <= 80 * 1024 && t.BN() <= (npad > 16 ? npad : 16);
}

// Shapes with the weight fragments in an LDS ring (bf16, one K partition),
// largest first.  (The 64x64 ring shape, 4 MFMAs per wave between barriers,
// measured slower than the register-weight kernel and is not chosen.)
static const int kPreferRing[] = {20, 24, 22, 21, 25, 23};

// 128x128 register-weight tiles, 4-chunk channel blocks.
static const int kWideHaloTile = 14;

// Tile shape of a conv for this state.  Deterministic: it depends on the
// layer, the batch and the chunk size only (never on a call's n), so every
// call of a state -- replayed or direct, chunked or offline -- runs the same
// arithmetic.  The arithmetic itself (K partitions, channel block) depends on
// the layer and the batch class only, never on the chunk size: a state built
// for another chunk size, or an offline state holding a whole utterance,
// computes the same bits.  First the K partitions: 4 (waves split K) for the
// streaming class (batch below DC_BATCHED_MIN), whose calls leave too few
// output tiles to fill the machine, else 1.  Then the channel block:
// as wide as the layer's channels (capped at 4 chunks for unsplit tiles),
// so no K step is padding.  Then the tile: for split K the largest that still
// gives the launch about three waves per SIMD, otherwise the first in
// preference order that keeps enough blocks.
static int pick_variant(const dc_state* s, const ConvOp& op)
{
    const int64_t B = s->cfg.batch;
    const int64_t F = (int64_t)s->cfg.chunk_tokens * s->fpt[op.level_in];
    const int nv = num_tile_variants();
    if (s->cfg.tile_variant > 0) {
        // a forced shape that does not fit this layer falls back to the largest
        // fitting shape with the same arithmetic (K partitions, channel block)
        const int fv = s->cfg.tile_variant - 1;
        if (variant_fits(op, fv)) return fv;
        int best = -1;
        for (int v = 0; v < nv; v++)
            if (tile_variant(v).WGK == tile_variant(fv).WGK && tile_variant(v).KCH == tile_variant(fv).KCH &&
                variant_fits(op, v) && (best < 0 || tile_variant(v).BM() * tile_variant(v).BN() >
                                                        tile_variant(best).BM() * tile_variant(best).BN()))
                best = v;
        if (best >= 0) return best;
    }
    auto blocks = [&](const TileShape& t) {
        return B * ((F + t.BM() - 1) / t.BM()) * ((op.N + t.BN() - 1) / t.BN());
    };
    // a resblock conv shares its launch with the parallel branches' convs:
    // the launch has that many times the blocks (the K-partition choice
    // below still looks at one conv)
    const int64_t members = op.stage >= 0 ? s->cfg.n_rb : 1;
    // the branch-mean position: the other branches' last convs share one
    // launch and the mean conv runs alone, so those launches have fewer blocks
    // than `members` counts (the shapes it picks for them measured best anyway)
    const bool mean_pos = op.stage >= 0 && op.half == 2 && op.dil_i == s->cfg.n_dil - 1 && s->cfg.n_rb > 1;
    auto eff = [&](const TileShape& t) {
        const int bm = t.BM();
        return (double)F / (double)(((F + bm - 1) / bm) * bm);
    };
    const int kq = op.bf16 ? 32 : 16;
    const int kch_all = (op.Ci + kq - 1) / kq;      // chunks covering every input channel
    const int wgk = B < DC_BATCHED_MIN ? 4 : 1;
    // channel-block candidates, widest first: no wider than the channels
    // (nor than 4 chunks when waves do not split K)
    for (int kch = 32; kch >= 1; kch /= 2) {
        if (kch > kch_all && kch > 1) continue;
        if (wgk == 1 && kch > 4) continue;
        // fp32 resblock convs of the streaming class: channel blocks of at
        // most 128 channels.  The 256-channel stage's widest tile then stages
        // 34 KB instead of 68 KB, four blocks fit a CU instead of two, and its
        // grouped launches run in about one round of blocks instead of two.
        if (wgk == 4 && !op.bf16 && op.stage >= 0 && kch > 8) continue;
        // fp32 K-split convs of 256 channels or more with a 50-row left
        // context (the 256-channel stage at dilation 5): 16x32 tiles, so the
        // 66 staged rows serve 32 columns per block instead of 16 (the
        // grouped launch measured 24.9 -> 21.7 us; the 128-channel stage's
        // 32x32 tiles stay, where 16x32 measured slower)
        if (wgk == 4 && !op.bf16 && op.Ci >= 256 && (op.k - 1) * op.d >= 50) {
            for (int v = 0; v < nv; v++) {
                const TileShape t = tile_variant(v);
                if (t.WGK == 4 && t.KCH == kch && t.MB == 1 && t.NB == 2 && t.WGM == 1 && t.WGN == 1 && variant_fits(op, v))
                    return v;
            }
        }
        // a wide left context ((k-1)*d >= 30 rows): 128x128 tiles, whose
        // 128 output rows dilute the halo every block stages (a 64-row tile
        // stages 1.8x its rows at k = 11, d = 5), as long as the launch keeps
        // at least 1024 of them
        if (wgk == 1 && (op.k - 1) * op.d >= 30) {
            const TileShape t = tile_variant(kWideHaloTile);
            if (t.KCH == kch && variant_fits(op, kWideHaloTile) && members * blocks(t) >= 1024 && eff(t) >= 0.75)
                return kWideHaloTile;
        }
        if (wgk == 1 && op.bf16 && !op.split && !(s->cfg.flags & DC_NO_RING)) {
            // the ring shapes first, for unsplit operands (split ones read their
            // low halves unprefetched there) and launches that keep the machine
            // busy for at least two rounds of blocks (two resident per CU; with
            // fewer the register-weight kernel measured faster), or one round
            // for a narrow left context (below 30 rows, where the ring's
            // staging is short: the B=16 256-channel convs at dilation 1, not
            // counting the branch-mean position's smaller launches): of those,
            // the one with the least padding in rows and columns (then the
            // largest)
            const int64_t min_ring = (op.k - 1) * op.d < 30 && !mean_pos ? 512 : 1024;
            int bestr = -1;
            double bestr_score = -1.0;
            for (int v : kPreferRing) {
                const TileShape t = tile_variant(v);
                if (t.KCH != kch || !variant_fits(op, v) || members * blocks(t) < min_ring) continue;
                const int bn = t.BN();
                const double col = (double)op.N / (double)(((op.N + bn - 1) / bn) * bn);
                const double score = eff(t) * col;
                if (score > bestr_score + 1e-9) {
                    bestr_score = score;
                    bestr = v;
                }
            }
            if (bestr >= 0 && bestr_score >= 0.7) return bestr;
        }
        int best = -1;
        double best_score = -1.0;
        const bool bytes_heavy = op.res >= 0 || op.N <= 64;
        const int* pref = bytes_heavy ? kPrefer64 : kPreferLarge;
        const int npref = bytes_heavy ? (int)(sizeof(kPrefer64) / sizeof(int)) : (int)(sizeof(kPreferLarge) / sizeof(int));
        const int* order = wgk == 4 ? nullptr : pref;
        for (int oi = 0; oi < (wgk == 4 ? nv : npref); oi++) {
            const int v = order ? order[oi] : oi;
            const TileShape t = tile_variant(v);
            if (t.WGK != wgk || t.KCH != kch || !variant_fits(op, v)) continue;
            double score;
            if (wgk == 4) {
                // waves of the whole launch (all its members) up to three per
                // SIMD, then larger tiles: each wave's operands then serve
                // more MFMAs and the layer's weights are read by fewer blocks
                const double waves = (double)(members * blocks(t)) * 4.0;
                score = (waves < 3072.0 ? waves : 3072.0) * eff(t) * (1.0 + 0.1 * std::log2((double)(t.MB * t.NB)));
            } else {
                // the first shape in preference order that keeps enough blocks
                // (a conv whose call fits in one row tile per stream -- the
                // pre-stack -- wants two rounds of them: at B=128 its 64x64
                // tiles measured 7% faster than 64x128 ones at 512 blocks)
                const int64_t min_blocks = !op.transposed && F <= t.BM() ? 1024 : 512;
                if (members * blocks(t) >= min_blocks && eff(t) >= 0.75) return v;
                score = (double)(members * blocks(t) < 512 ? members * blocks(t) : 512) * eff(t);
            }
            if (score > best_score) {
                best_score = score;
                best = v;
            }
        }
        if (best >= 0) return best;
    }
    // nothing with the preferred partitions: any fitting shape, unsplit first
    for (int v = 0; v < nv; v++)
        if (tile_variant(v).WGK == 1 && variant_fits(op, v)) return v;
    return 0;
}

// ------------------------------------------------------------ the network

static int add_ring(dc_state* s, const std::string& name, int C, int elem, int level)
{
    Ring r;
    r.C = C;
    r.elem = elem;
    r.level = level;
    s->rings.push_back(r);
    s->ring_names.push_back(name);
    s->ring_ctx.push_back(0);
    s->ring_onchip.push_back(false);
    return (int)s->rings.size() - 1;
}

static void need_ctx(dc_state* s, int ring, int ctx)
{
    if (ctx > s->ring_ctx[ring]) s->ring_ctx[ring] = ctx;
}

// Resblock pairs of a stage run fused (h on chip) for bf16 with enough
// streams to fill the machine, at the channel counts the fused kernel has
// shapes for, unless the caller forces a tile shape or asks for no fusion.
static bool fuse_stage(const dc_cfg& c, int channels)
{
    if (c.dtype != DC_BF16 || (c.flags & DC_NO_FUSE) || c.tile_variant != 0 || c.batch < DC_BATCHED_MIN)
        return false;
    int k_max = 1, d_max = 1;
    for (int j = 0; j < c.n_rb; j++) k_max = c.rb_kernel[j] > k_max ? c.rb_kernel[j] : k_max;
    for (int i = 0; i < c.n_dil; i++) d_max = c.dil[i] > d_max ? c.dil[i] : d_max;
    for (int v = 0; v < num_pair_variants(); v++)
        if (pair_variant(v).C() == channels)
            return pair_variant(v).fits(k_max, d_max) && pair_lds_bytes(v) <= 80 * 1024;
    return false;
}

static void build_network(dc_state* s)
{
    const dc_cfg& c = s->cfg;
    const bool bf = c.dtype == DC_BF16;
    const int opE = bf ? kBF16 : kF32;
    // the stages' residual stream (upsample output, resblock sums, stage
    // output): fp16 next to bf16 operands, fp32 otherwise
    const int opR = bf ? kF16 : kF32;
    size_t off = (size_t)c.vocab * c.embed;  // blob float offset after the embedding
    auto conv = [&](const std::string& name, int in, int out, int Ci, int N, int k, int d, int level) -> ConvOp& {
        ConvOp op;
        op.name = name;
        op.in = in;
        op.out = out;
        op.Ci = Ci;
        op.N = N;
        op.out_C = N;
        op.k = k;
        op.d = d;
        op.bf16 = bf;
        op.level_in = level;
        op.blob_w = off;
        off += (size_t)N * Ci * k;
        op.blob_b = off;
        off += (size_t)N;
        s->convs.push_back(op);
        return s->convs.back();
    };

    const int C0 = c.channels[0];
    s->ring_E = add_ring(s, "embed", C0, opE, 0);
    int cur = s->ring_E;
    for (int l = 0; l < c.n_pre; l++) {
        // pre-stack outputs stay fp32; a bf16 consumer takes them as hi + lo
        // operands (these layers carry most of the rounding sensitivity)
        const int P = add_ring(s, "pre" + std::to_string(l), C0, kF32, 0);
        ConvOp& op = conv("pre" + std::to_string(l), cur, P, C0, C0, c.pre_kernel, 1, 0);
        op.out_act = 1;
        op.split = bf && l > 0;
        need_ctx(s, cur, c.pre_kernel - 1);
        cur = P;
    }
    for (int st = 0; st < c.n_stages; st++) {
        const int ci = c.channels[st], co = c.channels[st + 1], u = c.up_rate[st];
        const std::string sn = "s" + std::to_string(st);
        const bool src_here = c.n_harmonics > 0 && st == c.n_stages - 1;
        if (src_here) s->ring_src = add_ring(s, "src", c.hop, kF32, st + 1);   // ctx 0: one call's samples
        const int Y = add_ring(s, sn + ".y", co, opR, st + 1);
        {
            ConvOp op;
            op.name = sn + ".up";
            op.in = cur;
            op.out = Y;
            op.Ci = ci;
            op.N = u * co;
            op.out_C = co;
            op.k = 2;
            op.d = 1;
            op.u = u;
            op.transposed = true;
            op.in_act = 1;
            op.bf16 = bf;
            op.split = bf;
            op.level_in = st;
            op.blob_w = off;
            off += (size_t)ci * co * 2 * u;
            op.blob_b = off;
            off += (size_t)co;
            if (src_here) op.src_ring = s->ring_src;
            s->convs.push_back(op);
            need_ctx(s, cur, 1);
        }
        std::vector<int> zlast;
        int X = -1;
        const bool fuse = fuse_stage(c, co);
        for (int j = 0; j < c.n_rb; j++) {
            const int kj = c.rb_kernel[j];
            int zin = Y;
            for (int i = 0; i < c.n_dil; i++) {
                const std::string pn = sn + ".rb" + std::to_string(j);
                const int H = add_ring(s, pn + ".h" + std::to_string(i), co, opE, st + 1);
                {
                    ConvOp& op = conv(pn + ".d" + std::to_string(i) + ".c1", zin, H, co, co, kj, c.dil[i], st + 1);
                    op.in_act = 1;
                    op.out_act = 1;
                    op.stage = st;
                    op.branch = j;
                    op.dil_i = i;
                    op.half = 1;
                    // fused: the pair reads z back far enough for both convs
                    need_ctx(s, zin, (kj - 1) * c.dil[i] + (fuse ? kj - 1 : 0));
                }
                if (fuse) {
                    s->ring_onchip[H] = true;
                    s->convs.back().partner = (int)s->convs.size();
                }
                const bool last = i == c.n_dil - 1;
                int Z;
                if (last && j == c.n_rb - 1)
                    Z = X = add_ring(s, sn + ".x", co, opR, st + 1);
                else
                    Z = add_ring(s, pn + ".z" + std::to_string(i), co, opR, st + 1);
                ConvOp& op = conv(pn + ".d" + std::to_string(i) + ".c2", H, Z, co, co, kj, 1, st + 1);
                op.res = zin;
                op.stage = st;
                op.branch = j;
                op.dil_i = i;
                op.half = 2;
                if (fuse) op.partner = (int)s->convs.size() - 2;
                need_ctx(s, H, kj - 1);
                if (Z == X) {
                    op.n_mean = (int)zlast.size();
                    for (int m = 0; m < op.n_mean; m++) op.mean[m] = zlast[m];
                }
                zin = Z;
            }
            zlast.push_back(zin);
        }
        cur = X;
    }
    const int L = c.n_stages;
    const int hc = 2 * (c.n_fft / 2 + 1);
    s->ring_S = add_ring(s, "head", hc, kF32, L);
    {
        ConvOp& op = conv("head", cur, s->ring_S, c.channels[L], hc, c.head_kernel, 1, L);
        op.in_act = 1;
        // bf16 weights are exact in bf16, and the fp32 operand is carried as a
        // hi + lo pair: the head keeps (nearly) fp32 products on bf16 MFMA
        op.split = bf;
        need_ctx(s, cur, c.head_kernel - 1);
    }
    s->ring_G = add_ring(s, "G", c.n_fft, kF32, L);
    need_ctx(s, s->ring_G, c.n_fft / c.hop - 1);
}

// The launch schedule of a chunk step.  Resblock convs at the same position
// (stage, dilation, first or second conv) of the parallel branches run as
// one launch; the branch-mean conv runs after the other branches' last convs
// it reads.  Members share the tile shape of the member with the widest left
// context (their arithmetic is the same: K partitions and channel block
// depend only on the channels).
// Fused-pair shape for a channel count: for 64 channels the 128-frame
// block (more reuse of each weight fragment), else the one shape there is.
#ifndef DC_PAIR64_VARIANT
#define DC_PAIR64_VARIANT 1
#endif
static int pair_shape_for(int channels)
{
    if (channels == 64) return DC_PAIR64_VARIANT;
    for (int v = 0; v < num_pair_variants(); v++)
        if (pair_variant(v).C() == channels) return v;
    return 0;
}

static void build_schedule(dc_state* s)
{
    const dc_cfg& c = s->cfg;
    s->launches.push_back({L_EMBED, {}, "embed"});
    if (c.n_harmonics > 0) {
        s->launches.push_back({L_PHASE, {}, "src.phase"});
        s->launches.push_back({L_SOURCE, {}, "src"});
    }
    auto add_group = [&](std::vector<int> m, const std::string& name) {
        int widest = m[0];
        for (int i : m)
            if ((s->convs[i].k - 1) * s->convs[i].d > (s->convs[widest].k - 1) * s->convs[widest].d) widest = i;
        const TileShape tw = tile_variant(s->convs[widest].variant);
        bool same = true;
        for (int i : m) {
            const TileShape ti = tile_variant(s->convs[i].variant);
            same = same && ti.WGK == tw.WGK && ti.KCH == tw.KCH;
        }
        if (!same || m.size() > (size_t)kMaxGroup) {
            for (int i : m) s->launches.push_back({L_CONV, {i}, s->convs[i].name});
            return;
        }
        for (int i : m) s->convs[i].variant = s->convs[widest].variant;
        // members with the most taps first: their blocks are the longest, and
        // blocks are dispatched in member order (when a launch has more blocks
        // than the machine holds, the long ones must not start last)
        // (batched tiles only: with K split across waves, at batch 1, the
        // branch order measured faster)
        if (tw.WGK == 1)
            std::stable_sort(m.begin(), m.end(), [&](int a, int b) { return s->convs[a].k > s->convs[b].k; });
        s->launches.push_back({L_CONV, m, name});
    };
    const int nconv = (int)s->convs.size();
    int i = 0;
    while (i < nconv) {
        const ConvOp& op = s->convs[i];
        if (op.stage < 0) {
            s->launches.push_back({L_CONV, {i}, op.name});
            i++;
            continue;
        }
        const int st = op.stage;
        std::vector<int> region;
        while (i < nconv && s->convs[i].stage == st) region.push_back(i++);
        const std::string sn = "s" + std::to_string(st);
        if (s->convs[region[0]].partner >= 0) {
            // fused pairs: one launch per dilation position (members: the
            // branches' first convs); the branch-mean pair runs last, alone
            const int pv = pair_shape_for(s->convs[region[0]].Ci);
            for (int di = 0; di < c.n_dil; di++) {
                std::vector<int> m;
                for (int j = 0; j < c.n_rb; j++)
                    for (int r : region)
                        if (s->convs[r].branch == j && s->convs[r].dil_i == di && s->convs[r].half == 1) m.push_back(r);
                const std::string pos = ".d" + std::to_string(di) + ".pair";
                Launch la{L_PAIR, {}, "", pv};
                // members with the most taps first: their blocks are the longest,
                // and blocks are dispatched in member order
                auto by_taps = [&](std::vector<int>& v) {
                    std::stable_sort(v.begin(), v.end(), [&](int a, int b) { return s->convs[a].k > s->convs[b].k; });
                };
                if (di == c.n_dil - 1 && c.n_rb > 1) {
                    la.convs.assign(m.begin(), m.end() - 1);
                    by_taps(la.convs);
                    la.name = sn + ".rb<" + std::to_string(c.n_rb - 1) + pos;
                    s->launches.push_back(la);
                    la.convs = {m.back()};
                    la.name = sn + ".rb" + std::to_string(c.n_rb - 1) + pos + ".mean";
                    s->launches.push_back(la);
                } else {
                    la.convs = m;
                    by_taps(la.convs);
                    la.name = sn + ".rb*" + pos;
                    s->launches.push_back(la);
                }
            }
            continue;
        }
        for (int di = 0; di < c.n_dil; di++)
            for (int half = 1; half <= 2; half++) {
                std::vector<int> m;
                for (int j = 0; j < c.n_rb; j++)
                    for (int r : region)
                        if (s->convs[r].branch == j && s->convs[r].dil_i == di && s->convs[r].half == half) m.push_back(r);
                const std::string pos = ".d" + std::to_string(di) + ".c" + std::to_string(half);
                const bool mean = half == 2 && di == c.n_dil - 1 && c.n_rb > 1;
                if (!mean) {
                    add_group(m, sn + ".rb*" + pos);
                } else {
                    add_group(std::vector<int>(m.begin(), m.end() - 1), sn + ".rb<" + std::to_string(c.n_rb - 1) + pos);
                    add_group({m.back()}, sn + ".rb" + std::to_string(c.n_rb - 1) + pos + ".mean");
                }
            }
    }
    s->launches.push_back({L_ISTFT, {}, "istft"});   // also advances the clock
}

// ------------------------------------------------------------ one chunk step
//
// A step is a fixed list of launches ("layers"): 0 embed, 1..C the convs in
// network order, then the iSTFT tail (spectrum, iDFT, window, overlap-add)
// and the clock.

static int layer_count(const dc_state* s) { return (int)s->launches.size(); }

static ConvParams conv_params(const dc_state* s, const ConvOp& op, int n)
{
    const dc_cfg& c = s->cfg;
    const Ring& in = s->rings[op.in];
    const Ring& out = s->rings[op.out];
    ConvParams p{};
    p.in = in.ptr;
    p.in_R = in.R;
    p.in_C = in.C;
    p.in_elem = in.elem;
    p.in_act = op.in_act;
    p.split = op.split;
    p.wp = s->arena + op.w_off;
    p.bias = (const float*)(s->arena + op.b_off);
    p.CB = op.CB;
    p.n_cb = op.n_cb;
    p.k = op.k;
    p.d = op.d;
    p.N = op.N;
    p.NB16 = op.NB16;
    p.out = out.ptr;
    p.out_R = out.R;
    p.out_C = out.C;
    p.out_elem = out.elem;
    p.out_act = op.out_act;
    p.u = op.u;
    if (op.res >= 0) {
        p.res = s->rings[op.res].ptr;
        p.res_R = s->rings[op.res].R;
    }
    p.n_mean = op.n_mean;
    for (int m = 0; m < op.n_mean; m++) {
        p.mean[m] = s->rings[op.mean[m]].ptr;
        p.mean_R = s->rings[op.mean[m]].R;
    }
    p.B = c.batch;
    p.F = (int)(n * s->fpt[op.level_in]);
    p.tiles_t = (p.F + tile_variant(op.variant).BM() - 1) / tile_variant(op.variant).BM();
    p.clock = s->clock;
    p.in_fpt = s->fpt[op.level_in];
    p.slope = c.lrelu_slope;
    p.err = s->err;
    if (op.src_ring >= 0) {
        p.src = (const float*)s->rings[op.src_ring].ptr;
        p.src_R = s->rings[op.src_ring].R;
        p.sd_w = (const float*)(s->arena + s->src_down_off);
        p.sd_b = p.sd_w + (size_t)op.out_C * c.hop;
    }
    return p;
}

// ptab: the per-call phase table (the arena's, or the static scratch of
// dc_decode_chunk_f0_static when non-null).
static SourceParams source_params(const dc_state* s, int n, double* ptab = nullptr)
{
    const dc_cfg& c = s->cfg;
    SourceParams p{};
    p.f0 = s->f0;
    p.carry = (double*)(s->arena + s->phase_off);
    p.tags = (int64_t*)(p.carry + (size_t)c.batch * 2 * (c.n_harmonics + 1));
    p.ptab = ptab ? ptab : (double*)(s->arena + s->ptab_off);
    p.src = (float*)s->rings[s->ring_src].ptr;
    p.src_R = s->rings[s->ring_src].R;
    p.mw = (const float*)(s->arena + s->src_w_off);
    p.mb = p.mw + c.n_harmonics + 1;
    p.B = c.batch;
    p.F0 = (int)(n * s->fpt[0]);
    p.H1 = c.n_harmonics + 1;
    p.S = (int)(s->fpt[c.n_stages] / s->fpt[0] * c.hop);
    p.fpt0 = s->fpt[0];
    p.fptL = s->fpt[c.n_stages];
    p.clock = s->clock;
    p.start = s->start;
    p.keys = s->keys;
    p.amp = c.sine_amp;
    p.noise = c.noise_std;
    p.thr = c.voiced_threshold;
    p.sr = (double)c.sample_rate;
    p.seed = c.rng_seed;
    return p;
}

#ifndef DC_PAIR_BLOCKS
#define DC_PAIR_BLOCKS 2048
#endif
static PairParams pair_params(const dc_state* s, const ConvOp& c1, int pv, int n, int members)
{
    const dc_cfg& c = s->cfg;
    const ConvOp& c2 = s->convs[c1.partner];
    const Ring& z = s->rings[c1.in];
    const Ring& o = s->rings[c2.out];
    PairParams p{};
    p.z = (const uint16_t*)z.ptr;
    p.z_R = z.R;
    p.w1 = s->arena + c1.w_off;
    p.b1 = (const float*)(s->arena + c1.b_off);
    p.w2 = s->arena + c2.w_off;
    p.b2 = (const float*)(s->arena + c2.b_off);
    p.out = (uint16_t*)o.ptr;
    p.out_R = o.R;
    p.k = c1.k;
    p.d = c1.d;
    p.C = c1.Ci;
    p.NB16 = c1.NB16;
    p.n_mean = c2.n_mean;
    for (int m = 0; m < c2.n_mean; m++) {
        p.mean[m] = (const uint16_t*)s->rings[c2.mean[m]].ptr;
        p.mean_R = s->rings[c2.mean[m]].R;
    }
    p.B = c.batch;
    p.F = (int)(n * s->fpt[c1.level_in]);
    p.tiles_t = (p.F + pair_variant(pv).BM() - 1) / pair_variant(pv).BM();
    // sub-tiles per block: about DC_PAIR_BLOCKS blocks per launch (every block
    // but the first of a stream recomputes k - 1 frames of h and reloads the
    // z frames left of its run, so fewer, longer blocks do less work; more
    // blocks balance the members' different tap counts over the machine)
    const int64_t want = DC_PAIR_BLOCKS;
    const int64_t units = (int64_t)p.B * p.tiles_t * members;
    p.seg_t = (int)std::max<int64_t>(1, std::min<int64_t>(p.tiles_t, units / want));
    p.segs = (p.tiles_t + p.seg_t - 1) / p.seg_t;
    p.clock = s->clock;
    p.start = s->start;
    p.in_fpt = s->fpt[c1.level_in];
    p.slope = c.lrelu_slope;
    p.err = s->err;
    return p;
}

// timing: a launch re-run on its own (dc_time_layers), which must leave the
// clock where it is.
static hipError_t launch_layer(dc_state* s, int i, int n, hipStream_t st, double* ptab = nullptr, bool timing = false)
{
    const dc_cfg& c = s->cfg;
    const int L = c.n_stages;
    const int FL = (int)(n * s->fpt[L]);
    const Launch& la = s->launches[i];
    switch (la.kind) {
    case L_EMBED:
        return launch_embed(s->tok, n, c.batch, s->emb, c.vocab, c.embed, s->rings[s->ring_E].elem,
                            c.frames_per_token, s->rings[s->ring_E], s->clock, s->err, st);
    case L_CONV: {
        ConvParams ps[kMaxGroup];
        const int cnt = (int)la.convs.size();
        for (int m = 0; m < cnt; m++) ps[m] = conv_params(s, s->convs[la.convs[m]], n);
        const ConvOp& op = s->convs[la.convs[0]];
        return launch_conv(op.variant, op.bf16, ps, cnt, st);
    }
    case L_PAIR: {
        PairParams ps[kMaxGroup];
        const int cnt = (int)la.convs.size();
        for (int m = 0; m < cnt; m++) ps[m] = pair_params(s, s->convs[la.convs[m]], la.pair_variant, n, cnt);
        return launch_pair(la.pair_variant, ps, cnt, st);
    }
    case L_PHASE:
        return launch_phase(source_params(s, n, ptab), st);
    case L_SOURCE:
        return launch_source(source_params(s, n, ptab), st);
    case L_ISTFT:
        return launch_istft((const float*)s->rings[s->ring_S].ptr, s->rings[s->ring_S].R, c.batch, FL, s->table,
                            s->rings[s->ring_G], s->audio, s->clock, s->fpt[L], timing ? 0 : n, s->arrivals, st);
    default:
        return hipErrorInvalidValue;
    }
}

// With a harmonic source, its phase and source launches depend only on the
// call's f0, the clock and their own carry: they run on the side stream
// beside the pre-stack and the first stages, and the main stream waits for
// them just before the launch that adds the source (in a captured graph the
// fork and the join become two parallel branches).
static hipError_t enqueue_step(dc_state* s, int n, hipStream_t st, double* ptab = nullptr)
{
    hipError_t e = hipSuccess;
    if (s->side) {
        e = hipEventRecord(s->fork_ev, st);
        if (e == hipSuccess) e = hipStreamWaitEvent(s->side, s->fork_ev, 0);
    }
    for (int i = 0; i < layer_count(s) && e == hipSuccess; i++) {
        const LaunchKind k = s->launches[i].kind;
        const bool on_side = s->side && (k == L_PHASE || k == L_SOURCE);
        if (s->side && i == s->src_join) e = hipStreamWaitEvent(st, s->join_ev, 0);
        if (e == hipSuccess) e = launch_layer(s, i, n, on_side ? s->side : st, ptab);
        if (e == hipSuccess && on_side && k == L_SOURCE) e = hipEventRecord(s->join_ev, s->side);
    }
    return e;
}

static hipError_t zero_state(dc_state* s)
{
    hipError_t e = hipMemsetAsync(s->arena + s->ring_begin, 0, s->ring_end - s->ring_begin, s->stream);
    if (e != hipSuccess) return e;
    e = hipMemsetAsync(s->clock, 0, sizeof(int64_t), s->stream);
    if (e != hipSuccess) return e;
    e = hipMemsetAsync(s->start, 0, (size_t)s->cfg.batch * sizeof(int64_t), s->stream);
    if (e != hipSuccess) return e;
    e = launch_init_keys(s->keys, s->cfg.batch, s->stream);
    if (e != hipSuccess) return e;
    e = hipMemsetAsync(s->arrivals, 0, sizeof(unsigned), s->stream);
    if (e != hipSuccess) return e;
    return hipMemsetAsync(s->err, 0, sizeof(int), s->stream);
}

// ------------------------------------------------------------------ the ABI

extern "C" {

// Both sizes read the stage and branch tables only as far as a valid
// configuration's counts reach: 0 for an invalid one.
int64_t dc_samples_per_token(const dc_cfg* cfg) { return cfg && validate(cfg).empty() ? samples_per_token(cfg) : 0; }

int64_t dc_blob_floats(const dc_cfg* cfg) { return cfg && validate(cfg).empty() ? blob_floats(cfg) : 0; }

static hipError_t static_scratch(int dev, void** out);

dc_status dc_init(const void* weights_blob, size_t blob_bytes, const dc_cfg* cfg, dc_state** out)
{
    if (!out) return fail(nullptr, DC_EINVAL, "out is NULL");
    *out = nullptr;
    if (!cfg || !weights_blob) return fail(nullptr, DC_EINVAL, "cfg or weights is NULL");
    if (cfg->abi_version != DC_ABI_VERSION) return fail(nullptr, DC_EVERSION, "abi_version mismatch");
    const std::string why = validate(cfg);
    if (!why.empty()) return fail(nullptr, DC_EINVAL, why);
    if (blob_bytes != (size_t)blob_floats(cfg) * sizeof(float))
        return fail(nullptr, DC_EINVAL, "blob size does not match the architecture");

    const auto t_start = std::chrono::steady_clock::now();
    dc_state* s = new dc_state();
    s->cfg = *cfg;
    const dc_cfg& c = s->cfg;
    const bool bf = c.dtype == DC_BF16;
    s->fpt[0] = c.frames_per_token;
    for (int i = 0; i < c.n_stages; i++) s->fpt[i + 1] = s->fpt[i] * c.up_rate[i];
    s->spt = samples_per_token(&c);
    build_network(s);
    for (auto& op : s->convs) {
        op.variant = pick_variant(s, op);
        if (op.partner >= 0) {
            // a fused pair's convs are packed for one partition and a channel
            // block of all their channels, the arithmetic of the pair kernel
            for (int v = 0; v < num_tile_variants(); v++)
                if (tile_variant(v).WGK == 1 && tile_variant(v).KCH * 32 == op.Ci) {
                    op.variant = v;
                    break;
                }
        }
        set_blocks(op);
    }
    build_schedule(s);

    // ---- arena layout: constants and weights, then rings, then I/O buffers
    const float* blob = (const float*)weights_blob;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    s->emb_off = take((size_t)c.vocab * c.embed * (bf ? 2 : 4));
    s->table_off = take(2 * 16 * 9 * sizeof(float));
    for (auto& op : s->convs) {
        op.w_off = take(op.w_bytes);
        op.b_off = take((size_t)op.N * sizeof(float));
    }
    const int CL = c.channels[c.n_stages];
    if (c.n_harmonics > 0) {
        s->src_w_off = take((size_t)(c.n_harmonics + 2) * sizeof(float));
        s->src_down_off = take((size_t)CL * (c.hop + 1) * sizeof(float));
    }
    const size_t weights_end = off;
    s->ring_begin = off;
    int64_t carry = 0;
    for (size_t i = 0; i < s->rings.size(); i++) {
        Ring& r = s->rings[i];
        r.ctx = s->ring_onchip[i] ? 0 : s->ring_ctx[i];
        r.R = s->ring_onchip[i] ? 0 : r.ctx + (int64_t)c.max_tokens * s->fpt[r.level];
        const size_t es = elem_bytes(r.elem);
        r.ptr = (void*)take((size_t)c.batch * r.R * r.C * es);  // offset for now
        carry += (int64_t)c.batch * r.ctx * r.C * es;
    }
    if (c.n_harmonics > 0) {
        // the carried phases sit with the rings: a reset zeroes them (a
        // stream at its first frame starts from its initial phases anyway)
        const size_t pb = (size_t)c.batch * 2 * (c.n_harmonics + 1) * sizeof(double) +
                          (size_t)c.batch * 2 * sizeof(int64_t);
        s->phase_off = take(pb);
        carry += (int64_t)pb;
    }
    s->ring_end = off;
    if (c.n_harmonics > 0) {
        s->ptab_off = take((size_t)c.batch * c.max_tokens * s->fpt[0] * (c.n_harmonics + 1) * sizeof(double));
        s->f0_off = take((size_t)c.batch * c.max_tokens * s->fpt[0] * sizeof(float));
    }
    s->tok_off = take((size_t)c.batch * c.max_tokens * sizeof(int32_t));
    s->audio_off = take((size_t)c.batch * c.max_tokens * s->spt * sizeof(float));
    s->clock_off = take(sizeof(int64_t));
    s->start_off = take((size_t)c.batch * sizeof(int64_t));
    s->keys_off = take((size_t)c.batch * sizeof(uint64_t));
    s->err_off = take(sizeof(int));
    s->arrivals_off = take(sizeof(unsigned));
    s->arena_bytes = off;

    hipError_t e = hipMalloc((void**)&s->arena, s->arena_bytes);
    if (e != hipSuccess) {
        delete s;
        return fail(nullptr, DC_ENOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    for (auto& r : s->rings) r.ptr = s->arena + (size_t)r.ptr;
    s->emb = s->arena + s->emb_off;
    s->table = (float*)(s->arena + s->table_off);
    s->tok = (int32_t*)(s->arena + s->tok_off);
    s->audio = (float*)(s->arena + s->audio_off);
    s->clock = (int64_t*)(s->arena + s->clock_off);
    s->start = (int64_t*)(s->arena + s->start_off);
    s->keys = (uint64_t*)(s->arena + s->keys_off);
    s->err = (int*)(s->arena + s->err_off);
    s->arrivals = (unsigned*)(s->arena + s->arrivals_off);
    if (c.n_harmonics > 0) s->f0 = (float*)(s->arena + s->f0_off);

    if (c.hip_stream) {
        s->stream = (hipStream_t)c.hip_stream;
    } else {
        e = hipStreamCreateWithFlags(&s->stream, hipStreamNonBlocking);
        if (e != hipSuccess) {
            (void)hipFree(s->arena);
            delete s;
            return fail(nullptr, DC_EDEVICE, std::string("hipStreamCreate: ") + hipGetErrorString(e));
        }
        s->own_stream = true;
    }
    if (c.n_harmonics > 0) {
        for (int i = 0; i < (int)s->launches.size(); i++)
            if (s->launches[i].kind == L_CONV && s->convs[s->launches[i].convs[0]].src_ring >= 0) s->src_join = i;
        e = hipStreamCreateWithFlags(&s->side, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&s->fork_ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&s->join_ev, hipEventDisableTiming);
        if (e == hipSuccess && s->src_join < 0) e = hipErrorInvalidValue;
        if (e != hipSuccess) {
            const std::string m = std::string("dc_init: side stream: ") + hipGetErrorString(e);
            dc_free(s);
            return fail(nullptr, DC_EDEVICE, m);
        }
    }
    // the device of the arena; a decoder with a harmonic source also resolves
    // that device's static scratch address here (dc_decode_chunk_f0_static)
    e = hipGetDevice(&s->device);
    if (e == hipSuccess && c.n_harmonics > 0) {
        void* p = nullptr;
        e = static_scratch(s->device, &p);
        s->static_ptab = (double*)p;
    }
    if (e != hipSuccess) {
        const std::string m = std::string("static scratch: ") + hipGetErrorString(e);
        dc_free(s);
        return fail(nullptr, DC_EDEVICE, m);
    }

    // ---- host-side packing of weights and device-resident constants
    std::vector<char> host(weights_end, 0);
    if (bf) {
        uint16_t* et = (uint16_t*)(host.data() + s->emb_off);
        for (size_t i = 0; i < (size_t)c.vocab * c.embed; i++) et[i] = host_f2bf(blob[i]);
    } else {
        std::memcpy(host.data() + s->emb_off, blob, (size_t)c.vocab * c.embed * sizeof(float));
    }
    {
        // Real inverse DFT x[n] = (1/N)[X0 + (-1)^n X_{N/2} + 2 sum Re X cos - Im X sin],
        // times the periodic Hann window w[n], divided by the overlap-add
        // normaliser sum_m w^2[n - hop m]; all in double, rounded once.
        const int N = c.n_fft, nb = N / 2 + 1;
        double w[64];
        for (int n = 0; n < N; n++) w[n] = 0.5 - 0.5 * std::cos(2.0 * M_PI * n / N);
        double norm = 0.0;
        for (int n = N - 1; n >= 0; n -= c.hop) norm += w[n] * w[n];
        float* tr = (float*)(host.data() + s->table_off);
        float* ti = tr + N * nb;
        for (int n = 0; n < N; n++)
            for (int kk = 0; kk < nb; kk++) {
                const double a = 2.0 * M_PI * kk * n / N;
                const double f = (kk == 0 || kk == N / 2) ? 1.0 : 2.0;
                tr[n * nb + kk] = (float)(w[n] * f * std::cos(a) / N / norm);
                ti[n * nb + kk] = (kk == 0 || kk == N / 2) ? 0.0f : (float)(-w[n] * 2.0 * std::sin(a) / N / norm);
            }
    }
    for (auto& op : s->convs) {
        pack_weights(op, blob, bf, host.data() + op.w_off);
        float* bias = (float*)(host.data() + op.b_off);
        for (int n = 0; n < op.N; n++) bias[n] = round_param(blob[op.blob_b + (op.transposed ? n % op.out_C : n)], bf);
    }
    if (c.n_harmonics > 0) {
        // merge W [H1], merge b, then down W [CL][hop] and down b [CL]: the
        // blob's last tensors, in that order
        const size_t H1 = (size_t)c.n_harmonics + 1;
        const float* tail = blob + (blob_floats(&c) - (int64_t)(H1 + 1 + (size_t)CL * c.hop + CL));
        float* mw = (float*)(host.data() + s->src_w_off);
        for (size_t i = 0; i < H1 + 1; i++) mw[i] = round_param(tail[i], bf);
        float* dw = (float*)(host.data() + s->src_down_off);
        for (size_t i = 0; i < (size_t)CL * c.hop + CL; i++) dw[i] = round_param(tail[H1 + 1 + i], bf);
    }
    s->st.weight_bytes = (int64_t)weights_end;
    s->st.arena_bytes = (int64_t)s->arena_bytes;
    s->st.carry_bytes = carry;
    s->st.ring_bytes = (int64_t)(s->ring_end - s->ring_begin);
    s->st.kernels_per_step = (int32_t)s->launches.size();

    e = hipMemcpy(s->arena, host.data(), weights_end, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemsetAsync(s->arena + weights_end, 0, s->arena_bytes - weights_end, s->stream);
    // Warm-up: one direct step on zero tokens loads every code object before capture.
    if (e == hipSuccess) e = enqueue_step(s, c.chunk_tokens, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e == hipSuccess && !(c.flags & DC_NO_GRAPH)) {
        hipStream_t cs = nullptr;
        e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        // one class: the whole step for n tokens (its kernel arguments, the
        // clock advance included, are fixed by n)
        auto capture = [&](int n, hipGraph_t* g, hipGraphExec_t* x) {
            hipError_t ce = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
            if (ce != hipSuccess) return ce;
            const hipError_t le = enqueue_step(s, n, cs);
            ce = hipStreamEndCapture(cs, g);
            if (le != hipSuccess) return le;
            if (ce != hipSuccess) return ce;
            return hipGraphInstantiate(x, *g, nullptr, nullptr, 0);
        };
        if (e == hipSuccess) e = capture(c.chunk_tokens, &s->graph, &s->exec);
        if (e == hipSuccess) {
            size_t nodes = 0;
            if (hipGraphGetNodes(s->graph, nullptr, &nodes) == hipSuccess) s->st.graph_nodes = (int32_t)nodes;
            s->st.graph_classes = 1;
        }
        if (e == hipSuccess && (c.flags & DC_FLUSH_CATALOG)) {
            s->flush_graph.assign(c.chunk_tokens, nullptr);
            s->flush_exec.assign(c.chunk_tokens, nullptr);
            for (int n = 1; n < c.chunk_tokens && e == hipSuccess; n++) {
                e = capture(n, &s->flush_graph[n], &s->flush_exec[n]);
                if (e == hipSuccess) s->st.graph_classes++;
            }
        }
        if (cs) (void)hipStreamDestroy(cs);
    }
    if (e == hipSuccess) e = zero_state(s);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) {
        const std::string m = std::string("dc_init: ") + hipGetErrorString(e);
        dc_free(s);
        return fail(nullptr, DC_EDEVICE, m);
    }
    s->st.capture_ms =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    *out = s;
    return DC_OK;
}

// One call: admission, staging of tokens (and f0), replay or direct launch,
// staging of the PCM.  f0 is non-null exactly for a decoder with a source.
// static_ptab non-null: dc_decode_chunk_f0_static (direct launches whose phase
// table is the device's static scratch; never a graph replay).
static dc_status decode_call(dc_state* s, const int32_t* tokens, const float* f0, int32_t n, float* audio_out,
                             double* static_ptab = nullptr)
{
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned; call dc_reset");
    const dc_cfg& c = s->cfg;
    if (!tokens || !audio_out || (c.n_harmonics > 0 && !f0)) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "tokens, f0 or audio_out is NULL");
    }
    if (n <= 0) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "n must be positive");
    }
    if (n > c.max_tokens) {
        s->st.rejected++;
        return fail(s, DC_ERANGE, "n exceeds max_tokens");
    }
    const bool host = (c.flags & DC_HOST_PTRS) != 0;
    const size_t tok_bytes = (size_t)c.batch * n * sizeof(int32_t);
    const size_t pcm_bytes = (size_t)c.batch * n * s->spt * sizeof(float);
    if (host) {
        for (size_t i = 0; i < (size_t)c.batch * n; i++)
            if (tokens[i] < 0 || tokens[i] >= c.vocab) {
                s->st.rejected++;
                return fail(s, DC_ERANGE, "token id outside [0, vocab)");
            }
    }
    hipError_t e = hipSuccess;
    if (tokens != s->tok) {
        e = hipMemcpyAsync(s->tok, tokens, tok_bytes, host ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice,
                           s->stream);
        if (e != hipSuccess) return device_fail(s, e, "token staging");
        s->st.staged_tokens++;
    }
    if (c.n_harmonics > 0 && f0 != s->f0) {
        const size_t f0_bytes = (size_t)c.batch * n * s->fpt[0] * sizeof(float);
        e = hipMemcpyAsync(s->f0, f0, f0_bytes, host ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "f0 staging");
        s->st.staged_f0++;
    }
    if (static_ptab) {
        e = enqueue_step(s, n, s->stream, static_ptab);
        if (e != hipSuccess) return device_fail(s, e, "direct launch (static scratch)");
        s->st.direct_static++;
    } else if (n == c.chunk_tokens && s->exec) {
        e = hipGraphLaunch(s->exec, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "hipGraphLaunch");
        s->st.replays++;
    } else if (n < c.chunk_tokens && (size_t)n < s->flush_exec.size() && s->flush_exec[n]) {
        e = hipGraphLaunch(s->flush_exec[n], s->stream);
        if (e != hipSuccess) return device_fail(s, e, "hipGraphLaunch");
        s->st.replays++;
        s->st.replays_flush++;
    } else {
        e = enqueue_step(s, n, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "direct launch");
        if (n != c.chunk_tokens) s->st.direct_shape++;
        else s->st.direct_nograph++;
    }
    s->st.calls++;
    s->clock_host += n;
    if (audio_out != s->audio) {
        e = hipMemcpyAsync(audio_out, s->audio, pcm_bytes, host ? hipMemcpyDeviceToHost : hipMemcpyDeviceToDevice,
                           s->stream);
        if (e != hipSuccess) return device_fail(s, e, "audio staging");
        s->st.staged_audio++;
    }
    if (host) return dc_sync(s);
    return DC_OK;
}

dc_status dc_decode_chunk(dc_state* s, const int32_t* tokens, int32_t n, float* audio_out)
{
    if (!s) return DC_EINVAL;
    if (s->cfg.n_harmonics > 0) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "this decoder has a harmonic source: call dc_decode_chunk_f0");
    }
    return decode_call(s, tokens, nullptr, n, audio_out);
}

dc_status dc_decode_chunk_f0(dc_state* s, const int32_t* tokens, const float* f0, int32_t n, float* audio_out)
{
    if (!s) return DC_EINVAL;
    if (s->cfg.n_harmonics == 0) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "this decoder has no harmonic source: call dc_decode_chunk");
    }
    return decode_call(s, tokens, f0, n, audio_out);
}

// ------------------------------------------- the static-scratch entry point
//
// The one per-call scratch buffer of the step is the harmonic source's phase
// table: every sinusoid's phase at the start of each f0 frame of the call,
// written by the phase kernel and read by the source kernel.
// dc_decode_chunk_f0_static keeps it in this file-scope device array instead
// of the state's arena.  Each device holds its own copy of the array for the
// life of the process; its device address is resolved once per device (at
// the dc_init of the first state with a source on that device), and host code
// passes only that address to kernels, never the array's name.
constexpr size_t kStaticScratchBytes = (size_t)4 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of `scratch` on device dev, which must be current.
static hipError_t static_scratch(int dev, void** out)
{
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress((void**)&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

dc_status dc_decode_chunk_f0_static(dc_state* s, const int32_t* tokens, const float* f0, int32_t n,
                                    float* audio_out)
{
    if (!s) return DC_EINVAL;
    const dc_cfg& c = s->cfg;
    if (c.n_harmonics == 0) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "this decoder has no harmonic source: it has no per-call scratch to move");
    }
    if (n > 0 && n <= c.max_tokens) {
        const size_t need = (size_t)c.batch * n * s->fpt[0] * (c.n_harmonics + 1) * sizeof(double);
        if (need > kStaticScratchBytes) {
            s->st.rejected++;
            char m[160];
            std::snprintf(m, sizeof m, "the call's phase table needs %zu bytes, more than the %zu-byte static scratch",
                          need, kStaticScratchBytes);
            return fail(s, DC_ERANGE, m);
        }
    }
    if (!s->static_ptab) return fail(s, DC_EDEVICE, "static scratch address was not resolved at dc_init");
    return decode_call(s, tokens, f0, n, audio_out, s->static_ptab);
}

dc_status dc_sync(dc_state* s)
{
    if (!s) return DC_EINVAL;
    hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "hipStreamSynchronize");
    int flag = 0;
    e = hipMemcpy(&flag, s->err, sizeof(int), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return device_fail(s, e, "error flag read");
    if (flag) {
        s->poisoned = true;
        if (flag & kErrTokenId) return fail(s, DC_ERANGE, "token id outside [0, vocab) reached the device; call dc_reset");
        return fail(s, DC_ERANGE, "a value beyond the binary16 range reached the residual stream; call dc_reset");
    }
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned; call dc_reset");
    return DC_OK;
}

dc_status dc_reset(dc_state* s)
{
    if (!s) return DC_EINVAL;
    hipError_t e = zero_state(s);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_reset");
    s->poisoned = false;
    s->clock_host = 0;
    return DC_OK;
}

dc_status dc_reset_stream(dc_state* s, int32_t b)
{
    if (!s) return DC_EINVAL;
    if (b < 0 || b >= s->cfg.batch) return fail(s, DC_EINVAL, "stream index out of range");
    for (const Ring& r : s->rings) {
        const size_t es = elem_bytes(r.elem);
        const size_t per = (size_t)r.R * r.C * es;
        hipError_t e = hipMemsetAsync((char*)r.ptr + (size_t)b * per, 0, per, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "dc_reset_stream");
    }
    // fused pairs recompute h of the left context: frames before this point are zeros
    hipError_t e = launch_mark_start(s->start, s->keys, b, s->clock, 0, (uint64_t)b, s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_reset_stream");
    return DC_OK;
}

int32_t* dc_token_buffer(dc_state* s) { return s ? s->tok : nullptr; }

float* dc_audio_buffer(dc_state* s) { return s ? s->audio : nullptr; }

float* dc_f0_buffer(dc_state* s) { return s ? s->f0 : nullptr; }

// ------------------------------------------------------------ carry snapshots
//
// One stream's carry as host bytes: what the next call of that stream reads
// from the past (every ring's ctx frames, the source's phases) plus where the
// stream is (tokens since its start) and its generator key.  Importing it
// into any slot of a state with the same layout continues the stream there
// exactly: the frames go to the slots of the receiving state's own clock,
// and the stream's start is placed that many tokens back.

namespace {

struct SnapHeader {
    uint64_t magic;
    uint64_t fingerprint;
    int64_t position;   // tokens decoded since the stream's start
    uint64_t key;       // source-generator key
    uint64_t bytes;     // whole snapshot
    uint64_t reserved;
};
constexpr uint64_t kSnapMagic = 0x313050414e534344ull;   // "DCSNAP01" as little-endian bytes

// FNV-1a over what a snapshot's meaning depends on: the architecture, the
// arithmetic, the source, and every ring's geometry (a fused state keeps
// wider z contexts and no h frames, so its snapshots differ from an unfused
// one's).
uint64_t layout_fingerprint(const dc_state* s)
{
    uint64_t h = 1469598103934665603ull;
    auto mix = [&](int64_t v) {
        for (int i = 0; i < 8; i++) {
            h ^= (uint64_t)((v >> (8 * i)) & 0xff);
            h *= 1099511628211ull;
        }
    };
    const dc_cfg& c = s->cfg;
    mix(DC_ABI_VERSION);
    mix(c.vocab), mix(c.embed), mix(c.frames_per_token), mix(c.n_pre), mix(c.pre_kernel), mix(c.n_stages);
    for (int i = 0; i < c.n_stages; i++) mix(c.up_rate[i]);
    for (int i = 0; i <= c.n_stages; i++) mix(c.channels[i]);
    mix(c.n_rb);
    for (int i = 0; i < c.n_rb; i++) mix(c.rb_kernel[i]);
    mix(c.n_dil);
    for (int i = 0; i < c.n_dil; i++) mix(c.dil[i]);
    mix(c.head_kernel), mix(c.n_fft), mix(c.hop), mix(c.dtype), mix(c.n_harmonics);
    for (const Ring& r : s->rings) mix(r.C), mix(r.elem), mix(r.ctx), mix(r.level);
    return h;
}

size_t snapshot_bytes(const dc_state* s)
{
    size_t n = sizeof(SnapHeader);
    for (const Ring& r : s->rings) n += (size_t)r.ctx * r.C * (elem_bytes(r.elem));
    n += (size_t)(s->cfg.n_harmonics > 0 ? s->cfg.n_harmonics + 1 : 0) * sizeof(double);
    return n;
}

// Copy frames [f0, f0 + nf) of stream b of ring r (host <-> device), as two
// runs where the ring wraps.
hipError_t ring_frames(const dc_state* s, const Ring& r, int b, int64_t f0, int nf, char* host, bool to_host)
{
    const size_t es = elem_bytes(r.elem), row = (size_t)r.C * es;
    int64_t slot = f0 % r.R;
    if (slot < 0) slot += r.R;
    int done = 0;
    while (done < nf) {
        const int run = (int)std::min<int64_t>(nf - done, r.R - slot);
        char* dev = (char*)r.ptr + ((size_t)b * r.R + slot) * row;
        const hipError_t e = to_host ? hipMemcpy(host + done * row, dev, run * row, hipMemcpyDeviceToHost)
                                     : hipMemcpy(dev, host + done * row, run * row, hipMemcpyHostToDevice);
        if (e != hipSuccess) return e;
        done += run;
        slot = 0;
    }
    return hipSuccess;
}

}  // namespace

int64_t dc_carry_bytes(const dc_state* s) { return s ? (int64_t)snapshot_bytes(s) : 0; }

dc_status dc_carry_export(dc_state* s, int32_t b, void* host_out, size_t bytes)
{
    if (!s) return DC_EINVAL;
    if (b < 0 || b >= s->cfg.batch || !host_out) return fail(s, DC_EINVAL, "bad stream index or buffer");
    if (bytes != snapshot_bytes(s)) return fail(s, DC_EINVAL, "buffer size differs from dc_carry_bytes");
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned; call dc_reset");
    hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_carry_export");
    int64_t start = 0;
    uint64_t key = 0;
    e = hipMemcpy(&start, s->start + b, sizeof start, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(&key, s->keys + b, sizeof key, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return device_fail(s, e, "dc_carry_export");
    char* out = (char*)host_out;
    SnapHeader hd{kSnapMagic, layout_fingerprint(s), s->clock_host - start, key, (uint64_t)bytes, 0};
    std::memcpy(out, &hd, sizeof hd);
    size_t off = sizeof hd;
    for (const Ring& r : s->rings) {
        if (r.ctx == 0) continue;
        const int64_t end = s->clock_host * s->fpt[r.level];
        e = ring_frames(s, r, b, end - r.ctx, r.ctx, out + off, true);
        if (e != hipSuccess) return device_fail(s, e, "dc_carry_export");
        off += (size_t)r.ctx * r.C * (elem_bytes(r.elem));
    }
    if (s->cfg.n_harmonics > 0) {
        // the phases of the next call's first f0 frame: the slot tagged with it
        const int H1 = s->cfg.n_harmonics + 1;
        const double* carry = (const double*)(s->arena + s->phase_off);
        const int64_t* tags = (const int64_t*)(carry + (size_t)s->cfg.batch * 2 * H1);
        int64_t tg[2];
        e = hipMemcpy(tg, tags + 2 * b, sizeof tg, hipMemcpyDeviceToHost);
        const int sel = tg[0] == s->clock_host * s->fpt[0] ? 0 : 1;
        if (e == hipSuccess)
            e = hipMemcpy(out + off, carry + ((size_t)b * 2 + sel) * H1, H1 * sizeof(double), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return device_fail(s, e, "dc_carry_export");
        off += H1 * sizeof(double);
    }
    return DC_OK;
}

dc_status dc_carry_import(dc_state* s, int32_t b, const void* host_in, size_t bytes)
{
    if (!s) return DC_EINVAL;
    if (b < 0 || b >= s->cfg.batch || !host_in) return fail(s, DC_EINVAL, "bad stream index or buffer");
    if (bytes != snapshot_bytes(s)) return fail(s, DC_EINVAL, "snapshot size differs from dc_carry_bytes");
    SnapHeader hd;
    std::memcpy(&hd, host_in, sizeof hd);
    if (hd.magic != kSnapMagic || hd.bytes != bytes) return fail(s, DC_EINVAL, "not a carry snapshot");
    if (hd.fingerprint != layout_fingerprint(s))
        return fail(s, DC_EINVAL, "snapshot of a different architecture, dtype or ring layout");
    if (hd.position < 0) return fail(s, DC_EINVAL, "bad snapshot position");
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned; call dc_reset");
    hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_carry_import");
    // the stream's rings start clean, then take the carried frames
    for (const Ring& r : s->rings) {
        const size_t per = (size_t)r.R * r.C * (elem_bytes(r.elem));
        if (per) e = hipMemset((char*)r.ptr + (size_t)b * per, 0, per);
        if (e != hipSuccess) return device_fail(s, e, "dc_carry_import");
    }
    const char* in = (const char*)host_in;
    size_t off = sizeof hd;
    for (const Ring& r : s->rings) {
        if (r.ctx == 0) continue;
        const int64_t end = s->clock_host * s->fpt[r.level];
        e = ring_frames(s, r, b, end - r.ctx, r.ctx, const_cast<char*>(in + off), false);
        if (e != hipSuccess) return device_fail(s, e, "dc_carry_import");
        off += (size_t)r.ctx * r.C * (elem_bytes(r.elem));
    }
    if (s->cfg.n_harmonics > 0) {
        const int H1 = s->cfg.n_harmonics + 1;
        double* carry = (double*)(s->arena + s->phase_off);
        int64_t* tags = (int64_t*)(carry + (size_t)s->cfg.batch * 2 * H1);
        const int64_t tg[2] = {s->clock_host * s->fpt[0], -1};
        e = hipMemcpy(carry + (size_t)b * 2 * H1, in + off, H1 * sizeof(double), hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(tags + 2 * b, tg, sizeof tg, hipMemcpyHostToDevice);
        if (e != hipSuccess) return device_fail(s, e, "dc_carry_import");
    }
    // the stream started `position` tokens before this state's next call
    e = launch_mark_start(s->start, s->keys, b, s->clock, hd.position, hd.key, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_carry_import");
    return DC_OK;
}

dc_status dc_get_stats(const dc_state* s, dc_stats* out)
{
    if (!s || !out) return DC_EINVAL;
    *out = s->st;
    out->clock_tokens = s->clock_host;
    return DC_OK;
}

int32_t dc_tap_find(const dc_state* s, const char* name)
{
    if (!s || !name) return -1;
    for (size_t i = 0; i < s->ring_names.size(); i++)
        if (s->ring_names[i] == name) return (int32_t)i;
    return -1;
}

dc_status dc_tap_read(dc_state* s, int32_t tap, int32_t b, int64_t frame0, int32_t nframes, float* host_out,
                      int32_t* channels)
{
    if (!s || !host_out || tap < 0 || tap >= (int32_t)s->rings.size() || b < 0 || b >= s->cfg.batch ||
        nframes < 0)
        return fail(s, DC_EINVAL, "bad tap arguments");
    const Ring& r = s->rings[tap];
    if (channels) *channels = r.C;
    const int64_t end = s->clock_host * s->fpt[r.level];
    if (frame0 < end - r.R || frame0 + nframes > end) return fail(s, DC_ERANGE, "frames not held by the ring");
    hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "dc_tap_read");
    const size_t es = elem_bytes(r.elem);
    std::vector<char> row((size_t)r.C * es);
    for (int32_t f = 0; f < nframes; f++) {
        int64_t slot = (frame0 + f) % r.R;
        if (slot < 0) slot += r.R;
        e = hipMemcpy(row.data(), (char*)r.ptr + ((size_t)b * r.R + slot) * r.C * es, row.size(),
                      hipMemcpyDeviceToHost);
        if (e != hipSuccess) return device_fail(s, e, "dc_tap_read copy");
        for (int ch = 0; ch < r.C; ch++)
            host_out[(size_t)f * r.C + ch] =
                r.elem == kF32    ? ((float*)row.data())[ch]
                : r.elem == kF16 ? host_h2f(((uint16_t*)row.data())[ch])
                                 : host_bf2f(((uint16_t*)row.data())[ch]);
    }
    return DC_OK;
}

int32_t dc_layer_count(const dc_state* s) { return s ? layer_count(s) : 0; }

dc_status dc_layer_info_get(const dc_state* s, int32_t i, dc_layer_info* out)
{
    if (!s || !out || i < 0 || i >= layer_count(s)) return DC_EINVAL;
    const dc_cfg& c = s->cfg;
    std::memset(out, 0, sizeof *out);
    const int n = c.chunk_tokens;
    const double B = c.batch;
    const int L = c.n_stages;
    const double FL = (double)n * s->fpt[L];
    const Launch& la = s->launches[i];
    auto set = [&](const std::string& kernel) {
        std::snprintf(out->name, sizeof out->name, "%s", la.name.c_str());
        std::snprintf(out->kernel, sizeof out->kernel, "%s", kernel.c_str());
    };
    switch (la.kind) {
    case L_EMBED: {
        const Ring& E = s->rings[s->ring_E];
        const double es = elem_bytes(E.elem);
        const double F = (double)n * c.frames_per_token;
        set("dc::embed_kernel");
        out->bytes = B * n * 4 + B * n * c.embed * es + B * F * c.embed * es;
        break;
    }
    case L_CONV: {
        const ConvOp& op0 = s->convs[la.convs[0]];
        const TileShape t = tile_variant(op0.variant);
        if (t.W)
            set("dc::wconv_kernel<" + std::to_string(t.MB) + ", " + std::to_string(t.NB) + ", " +
                std::to_string(t.WGM) + ", " + std::to_string(t.WGN) + ", " + std::to_string(t.KCH) + ">");
        else
            set("dc::conv_kernel<" + std::string(op0.bf16 ? "true" : "false") + ", " + std::to_string(t.MB) + ", " +
                std::to_string(t.NB) + ", " + std::to_string(t.WGM) + ", " + std::to_string(t.WGN) + ", " +
                std::to_string(t.WGK) + ", " + std::to_string(t.KCH) + ">");
        for (int ci : la.convs) {   // the members' work and compulsory bytes add up
            const ConvOp& op = s->convs[ci];
            const double F = (double)n * s->fpt[op.level_in];
            const Ring& in = s->rings[op.in];
            const Ring& o = s->rings[op.out];
            out->rows = (int64_t)(B * F);
            out->cols = op.N;
            out->depth += (int64_t)op.k * op.Ci;
            out->flops += 2.0 * B * F * op.N * op.Ci * op.k;
            const double wes = op.bf16 ? 2 : 4;
            const double ies = elem_bytes(in.elem), oes = elem_bytes(o.elem);
            const double Fo = F * op.u;
            out->bytes += (double)op.N * op.Ci * op.k * wes + B * (F + (op.k - 1) * op.d) * op.Ci * ies +
                          B * Fo * o.C * oes + (op.res >= 0 ? B * Fo * o.C * oes : 0) + op.n_mean * B * Fo * o.C * oes;
        }
        break;
    }
    case L_PAIR: {
        const PairShape t = pair_variant(la.pair_variant);
        set("dc::pair_kernel<" + std::to_string(t.MB) + ", " + std::to_string(t.NB) + ", " + std::to_string(t.WGM) +
            ", " + std::to_string(t.WGN) + ", " + std::to_string(t.KCH) + ", " + std::to_string(t.LZ) + ", " +
            std::to_string(t.LH) + ">");
        for (int ci : la.convs) {   // both convs' work; z once, the output once, both weights (fp16 rings)
            const ConvOp& a = s->convs[ci];
            const ConvOp& b2 = s->convs[a.partner];
            const double F = (double)n * s->fpt[a.level_in];
            out->rows = (int64_t)(B * F);
            out->cols = a.N;
            out->depth += (int64_t)a.k * a.Ci + (int64_t)b2.k * b2.Ci;
            out->flops += 2.0 * B * F * a.N * a.Ci * a.k + 2.0 * B * F * b2.N * b2.Ci * b2.k;
            out->bytes += 2.0 * ((double)a.N * a.Ci * a.k + (double)b2.N * b2.Ci * b2.k) +
                          B * (F + (a.k - 1) * a.d + (a.k - 1)) * a.Ci * 2 + B * F * b2.N * 2 +
                          b2.n_mean * B * F * b2.N * 2;
        }
        break;
    }
    case L_PHASE: {
        const double F0 = (double)n * s->fpt[0], H1 = c.n_harmonics + 1;
        set("dc::phase_kernel");
        out->bytes = B * F0 * 4 + B * F0 * H1 * 8 + 2 * B * H1 * 8;
        break;
    }
    case L_SOURCE: {
        const double F0 = (double)n * s->fpt[0], H1 = c.n_harmonics + 1;
        set("dc::source_kernel");
        out->bytes = B * F0 * 4 + B * F0 * H1 * 8 + B * FL * c.hop * 4;
        break;
    }
    default:   // the iSTFT tail: head output in, PCM out, the 3-frame left context in and out, the clock
        set("dc::istft_kernel");
        out->bytes = B * FL * (2 * (c.n_fft / 2 + 1) + c.hop) * 4 + 2.0 * B * (c.n_fft / c.hop - 1) * c.n_fft * 4 + 16;
    }
    return DC_OK;
}

dc_status dc_time_layers(dc_state* s, int32_t reps, double* us_per_launch)
{
    if (!s || !us_per_launch || reps < 1) return fail(s, DC_EINVAL, "bad dc_time_layers arguments");
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned; call dc_reset");
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipError_t e = hipEventCreate(&e0);
    if (e == hipSuccess) e = hipEventCreate(&e1);
    const int nl = layer_count(s);
    for (int i = 0; i < nl && e == hipSuccess; i++) {   // re-runs leave the clock where it is
        e = launch_layer(s, i, s->cfg.chunk_tokens, s->stream, nullptr, true);   // warm
        if (e == hipSuccess) e = hipEventRecord(e0, s->stream);
        for (int r = 0; r < reps && e == hipSuccess; r++)
            e = launch_layer(s, i, s->cfg.chunk_tokens, s->stream, nullptr, true);
        if (e == hipSuccess) e = hipEventRecord(e1, s->stream);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        us_per_launch[i] = 1000.0 * ms / reps;
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (e != hipSuccess) return device_fail(s, e, "dc_time_layers");
    return DC_OK;
}

const char* dc_last_error(const dc_state* s) { return s ? s->msg.c_str() : g_init_error.c_str(); }

void dc_free(dc_state* s)
{
    if (!s) return;
    if (s->stream) (void)hipStreamSynchronize(s->stream);
    if (s->exec) (void)hipGraphExecDestroy(s->exec);
    if (s->graph) (void)hipGraphDestroy(s->graph);
    for (hipGraphExec_t x : s->flush_exec)
        if (x) (void)hipGraphExecDestroy(x);
    for (hipGraph_t g : s->flush_graph)
        if (g) (void)hipGraphDestroy(g);
    if (s->side) (void)hipStreamSynchronize(s->side);
    if (s->arena) (void)hipFree(s->arena);
    if (s->fork_ev) (void)hipEventDestroy(s->fork_ev);
    if (s->join_ev) (void)hipEventDestroy(s->join_ev);
    if (s->side) (void)hipStreamDestroy(s->side);
    if (s->own_stream && s->stream) (void)hipStreamDestroy(s->stream);
    delete s;
}

}  // extern "C"
