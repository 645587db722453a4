// Host runtime of the streaming flow-decoder chunk step: configuration
// checks, one device arena per state (weights, per-step constants, the
// stacked carry, per-call buffers), the launch sequence of one call, graph
// capture of the f_call-frame call, and the C ABI of dc_flow.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "dc_flow.h"
#include "flow_internal.h"

using namespace dcf;

namespace {

std::string g_flow_init_error;

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }
int round_up(int v, int q) { return (v + q - 1) / q * q; }

// Offsets (floats) of the tensors of the blob.
struct BlobMap {
    int64_t t1W, t1b, t2W, t2b, inW, inb;
    std::vector<int64_t> ada, qkvW, qkvb, oW, ob, fc1W, fc1b, fc2W, fc2b;
    int64_t block_stride;
    int64_t fadaW, outW, outb;
    int64_t total;
};

BlobMap blob_map(const dc_flow_cfg& c)
{
    const int64_t D = c.dim, M = c.n_mel, T = c.t_dim, H = c.mlp;
    BlobMap m{};
    int64_t o = 0;
    auto take = [&](int64_t n) {
        const int64_t at = o;
        o += n;
        return at;
    };
    m.t1W = take(D * T);
    m.t1b = take(D);
    m.t2W = take(D * D);
    m.t2b = take(D);
    m.inW = take(D * 4 * M);
    m.inb = take(D);
    const int64_t b0 = o;
    for (int l = 0; l < c.depth; l++) {
        m.ada.push_back(take(6 * D * D));
        take(6 * D);
        m.qkvW.push_back(take(3 * D * D));
        m.qkvb.push_back(take(3 * D));
        m.oW.push_back(take(D * D));
        m.ob.push_back(take(D));
        m.fc1W.push_back(take(H * D));
        m.fc1b.push_back(take(H));
        m.fc2W.push_back(take(D * H));
        m.fc2b.push_back(take(D));
    }
    m.block_stride = c.depth > 0 ? (o - b0) / c.depth : 0;
    m.fadaW = take(2 * D * D);
    take(2 * D);
    m.outW = take(M * D);
    m.outb = take(M);
    m.total = o;
    return m;
}

std::string validate(const dc_flow_cfg* c)
{
    if (c->n_mel < 8 || c->n_mel % 8 != 0 || c->n_mel > 1024) return "n_mel must be a multiple of 8 in [8, 1024]";
    if (c->heads < 1 || c->dim != 64 * c->heads) return "dim must be 64 * heads";
    if (c->dim > 512) return "dim must be <= 512";
    if (c->depth < 1) return "depth must be >= 1";
    if (c->mlp < 32 || c->mlp % 32 != 0) return "mlp must be a positive multiple of 32";
    if (c->t_dim < 2 || c->t_dim % 2 != 0 || c->t_dim > 1024) return "t_dim must be even, in [2, 1024]";
    if (c->n_steps < 1 || c->n_steps > 1000) return "n_steps must be in [1, 1000]";
    if (c->f_chunk < 1 || c->f_call < c->f_chunk) return "need 1 <= f_chunk <= f_call";
    if (c->f_retained < 0 || c->f_retained % c->f_chunk != 0) return "f_retained must be a multiple of f_chunk";
    if (c->f_retained / c->f_chunk > 6) return "f_retained / f_chunk must be <= 6";
    if (c->f_prompt < 1) return "f_prompt must be >= 1";
    if (c->f_call > 4096 || c->f_prompt > 4096) return "f_call and f_prompt must be <= 4096";
    if (c->batch < 1 || c->batch > 4096) return "batch must be in [1, 4096]";
    if (c->dtype != DC_F32 && c->dtype != DC_BF16) return "dtype must be DC_F32 or DC_BF16";
    if (c->flags & ~(uint32_t)(DC_HOST_PTRS | DC_NO_GRAPH)) return "unknown flags";
    return "";
}

}  // namespace

struct dc_flow_state {
    dc_flow_cfg cfg{};
    hipStream_t stream = nullptr;
    bool own_stream = false;
    bool bf = false;
    size_t esz = 4;              // bytes of an operand element
    char* arena = nullptr;
    size_t arena_bytes = 0;
    // per-step weights (operand type) and biases (fp32)
    void* w_in = nullptr;
    std::vector<void*> w_qkv, w_o, w_fc1, w_fc2;
    void* w_out = nullptr;
    float* b_in = nullptr;
    std::vector<float*> b_qkv, b_o, b_fc1, b_fc2;
    float* b_out = nullptr;
    // per-step constants
    float *mods = nullptr, *fmods = nullptr, *t = nullptr, *dt = nullptr, *silu_temb = nullptr;
    // stream state
    int64_t *hist = nullptr, *pos = nullptr;
    int* plen = nullptr;
    uint64_t* keys = nullptr;
    float* spk = nullptr;
    // carry
    void* carry = nullptr;
    int Pr = 0, Sl = 0, R = 0, Fr = 0;
    int64_t stream_stride = 0;
    // per-call buffers
    void *xin = nullptr, *a = nullptr, *o = nullptr, *u = nullptr, *q = nullptr;
    float *h = nullptr, *v = nullptr, *x = nullptr;
    float *mu_in = nullptr, *mel_out = nullptr, *cond_in = nullptr, *gather = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    std::vector<int> plen_host;
    std::vector<int64_t> hist_host;
    dc_flow_stats st{};
    bool poisoned = false;
    std::string msg;
};

namespace {

dc_status fail(dc_flow_state* s, dc_status code, const std::string& why)
{
    if (s) s->msg = why;
    else g_flow_init_error = why;
    return code;
}

dc_status device_fail(dc_flow_state* s, hipError_t e, const char* where)
{
    s->poisoned = true;
    return fail(s, DC_EDEVICE, std::string(where) + ": " + hipGetErrorString(e));
}

CarryRef carry_ref(const dc_flow_state* s, int i, int l)
{
    const dc_flow_cfg& c = s->cfg;
    CarryRef r;
    r.base = (char*)s->carry + ((size_t)(i * c.depth + l) * 4 * c.heads) * s->Fr * 64 * s->esz;
    r.stream_stride = s->stream_stride;
    r.Fr = s->Fr;
    r.Pr = s->Pr;
    r.Sl = s->Sl;
    r.R = s->R;
    r.hist = s->hist;
    r.plen = s->plen;
    return r;
}

// Per-launch timing: events recorded around each launch of a profiled call.
struct Recorder {
    std::vector<std::string> role;
    std::vector<double> flops, bytes;
    std::vector<int> mfma;
    std::vector<hipEvent_t> ev;   // two per launch
    size_t at = 0;
};

// The launches of one call over Bc streams from b0 with n frames per stream.
// With a recorder, each launch is bracketed by events and described (role,
// algorithmic flops and bytes), and the state advance is left out.
hipError_t enqueue_call(dc_flow_state* s, int b0, int Bc, int n, int prompt, const float* mu, const float* cond,
                        float* mel, hipStream_t st, int* count, Recorder* rec = nullptr)
{
    const dc_flow_cfg& c = s->cfg;
    const int bf = s->bf ? 1 : 0;
    const int D = c.dim, M = c.n_mel, NL = c.depth, NS = c.n_steps;
    const int rows = Bc * 2 * n, Fq = round_up(n, 64);
    int k = 0;
    hipError_t e;
    const double es = (double)s->esz;
    const int64_t ext_keys = [&] {   // keys attended by all the call's queries, summed over its streams
        int64_t t = 0;
        if (!rec) return t;
        for (int b = b0; b < b0 + Bc; b++)
            t += prompt ? n : std::min<int64_t>(s->hist_host[b], s->R) * c.f_chunk + s->plen_host[b] + n;
        return t;
    }();
    std::string role;
    double fl = 0, by = 0;
    int mf = 0;
    auto describe = [&](const char* r, double f, double b, int m) {
        role = r;
        fl = f;
        by = b;
        mf = m;
    };
    auto gemm_cost = [&](const char* r, int N, int K, double a_es, double out_es, bool reads_h) {
        describe(r, 2.0 * rows * N * K, (double)rows * K * a_es + (double)N * K * es + (double)N * 4 +
                                            (double)rows * N * out_es * (reads_h ? 2 : 1), 1);
    };
#define DCF_TRY(x)                                                           \
    do {                                                                     \
        if (rec) {                                                           \
            e = hipEventRecord(rec->ev[2 * rec->at], st);                    \
            if (e != hipSuccess) return e;                                   \
        }                                                                    \
        e = (x);                                                             \
        if (e != hipSuccess) return e;                                       \
        if (rec) {                                                           \
            e = hipEventRecord(rec->ev[2 * rec->at + 1], st);                \
            if (e != hipSuccess) return e;                                   \
            rec->role[rec->at] = role;                                       \
            rec->flops[rec->at] = fl;                                        \
            rec->bytes[rec->at] = by;                                        \
            rec->mfma[rec->at] = mf;                                         \
            rec->at++;                                                       \
        }                                                                    \
        k++;                                                                 \
    } while (0)

    AssembleParams ap{mu, cond, s->spk, s->x, s->xin, s->pos, s->keys, c.rng_seed, c.temperature, n, b0, Bc, M};
    describe("assemble", 0, (double)Bc * n * M * 4 * (cond ? 2 : 1) + (double)rows * 4 * M * es + (double)Bc * n * M * 4, 0);
    DCF_TRY(launch_assemble(ap, bf, st));
    for (int i = 0; i < NS; i++) {
        GemmParams g{};
        g.M = rows;
        g.n = n;
        g.b0 = b0;
        g.heads = c.heads;
        g.dim = D;
        g.Fq = Fq;
        g.prompt = prompt;
        g.q = s->q;
        auto plain = [&](const void* A) {
            g.A = A;
            g.ln_h = nullptr;
            g.ln_shift = g.ln_scale = nullptr;
        };
        auto normed = [&](const float* shift, const float* scale) {   // A = LN(h) * (1 + scale) + shift
            g.A = s->a;                                                // written there for calls of many rows
            g.ln_h = s->h;
            g.ln_shift = shift;
            g.ln_scale = scale;
        };
        // input projection
        plain(s->xin);
        g.W = s->w_in;
        g.bias = s->b_in;
        g.N = D;
        g.K = 4 * M;
        g.h = s->h;
        gemm_cost("gemm:in", D, 4 * M, es, 4, false);
        DCF_TRY(launch_gemm(g, E_H, bf, st));
        for (int l = 0; l < NL; l++) {
            const float* md = s->mods + ((size_t)i * NL + l) * 6 * D;
            const CarryRef cr = carry_ref(s, i, l);
            normed(md, md + D);
            g.W = s->w_qkv[l];
            g.bias = s->b_qkv[l];
            g.N = 3 * D;
            g.K = D;
            g.carry = cr;
            gemm_cost("gemm:qkv", 3 * D, D, 4, es, false);
            DCF_TRY(launch_gemm(g, E_QKV, bf, st));
            AttnParams at{s->q, Fq, cr, s->o, prompt, n, b0, c.heads, D, c.f_chunk};
            // per (stream, branch, head): n queries x its keys x 64, twice (scores, values)
            describe("attn", 4.0 * 2 * c.heads * 64 * (double)n * ext_keys,
                     2.0 * 2 * c.heads * 64 * (double)ext_keys * es + 2.0 * rows * D * es, 1);
            DCF_TRY(launch_attn(at, Bc, bf, st));
            plain(s->o);
            g.W = s->w_o[l];
            g.bias = s->b_o[l];
            g.N = D;
            g.K = D;
            g.gate = md + 2 * D;
            gemm_cost("gemm:o", D, D, es, 4, true);
            DCF_TRY(launch_gemm(g, E_RES, bf, st));
            normed(md + 3 * D, md + 4 * D);
            g.W = s->w_fc1[l];
            g.bias = s->b_fc1[l];
            g.N = c.mlp;
            g.K = D;
            g.out = s->u;
            gemm_cost("gemm:fc1", c.mlp, D, 4, es, false);
            DCF_TRY(launch_gemm(g, E_GELU, bf, st));
            plain(s->u);
            g.W = s->w_fc2[l];
            g.bias = s->b_fc2[l];
            g.N = D;
            g.K = c.mlp;
            g.gate = md + 5 * D;
            gemm_cost("gemm:fc2", D, c.mlp, es, 4, true);
            DCF_TRY(launch_gemm(g, E_RES, bf, st));
        }
        const float* fm = s->fmods + (size_t)i * 2 * D;
        normed(fm, fm + D);
        g.W = s->w_out;
        g.bias = s->b_out;
        g.N = M;
        g.K = D;
        g.out = s->v;
        gemm_cost("gemm:out", M, D, 4, 4, false);
        DCF_TRY(launch_gemm(g, E_VEL, bf, st));
        EulerParams ep{s->v, s->x, s->xin, i == NS - 1 ? mel : nullptr, s->dt + i, c.cfg_rate, n, Bc, M};
        describe("euler", 5.0 * Bc * n * M, (double)rows * M * 4 + 2.0 * Bc * n * M * 4 + (double)rows * M * es, 0);
        DCF_TRY(launch_euler(ep, bf, st));
    }
    describe("advance", 0, 0, 0);
    if (!prompt && n >= c.f_chunk && !rec)
        DCF_TRY(launch_advance(s->hist, s->pos, s->plen, 2, 0, 0, c.batch, c.f_chunk, st));
#undef DCF_TRY
    if (count) *count = k;
    return hipSuccess;
}

void host_advance(dc_flow_state* s, int n)
{
    if (n >= s->cfg.f_chunk)
        for (auto& h : s->hist_host) h++;
}

}  // namespace

extern "C" {

int64_t dc_flow_blob_floats(const dc_flow_cfg* cfg)
{
    if (!cfg || !validate(cfg).empty()) return 0;
    return blob_map(*cfg).total;
}

dc_status dc_flow_init(const void* weights_blob, size_t blob_bytes, const dc_flow_cfg* cfg, dc_flow_state** out)
{
    if (!out) return fail(nullptr, DC_EINVAL, "out is NULL");
    *out = nullptr;
    if (!cfg || !weights_blob) return fail(nullptr, DC_EINVAL, "cfg or weights is NULL");
    if (cfg->abi_version != DC_FLOW_ABI_VERSION) return fail(nullptr, DC_EVERSION, "abi_version mismatch");
    const std::string why = validate(cfg);
    if (!why.empty()) return fail(nullptr, DC_EINVAL, why);
    const BlobMap bm = blob_map(*cfg);
    if (blob_bytes != (size_t)bm.total * sizeof(float))
        return fail(nullptr, DC_EINVAL, "blob size does not match the architecture");

    const auto t_start = std::chrono::steady_clock::now();
    dc_flow_state* s = new dc_flow_state();
    s->cfg = *cfg;
    const dc_flow_cfg& c = s->cfg;
    s->bf = c.dtype == DC_BF16;
    s->esz = s->bf ? 2 : 4;
    const int D = c.dim, M = c.n_mel, NL = c.depth, NS = c.n_steps, B = c.batch;
    const float* blob = (const float*)weights_blob;
    s->plen_host.assign(B, 0);   // no stream has a turn
    s->hist_host.assign(B, 0);

    // carry geometry: prompt region and slots padded to 4 frames (aligned
    // 4-key value groups), R history slots plus the one a call writes
    s->Pr = round_up(c.f_prompt, 4);
    s->Sl = round_up(c.f_call, 4);
    s->R = c.f_retained / c.f_chunk;
    s->Fr = s->Pr + (s->R + 1) * s->Sl;
    s->stream_stride = (int64_t)NS * NL * 4 * c.heads * s->Fr * 64;

    // arena layout
    size_t off = 0;
    auto place = [&](size_t bytes) {
        const size_t at = off;
        off = align256(off + bytes);
        return at;
    };
    const size_t es = s->esz;
    const size_t o_win = place((size_t)D * 4 * M * es);
    std::vector<size_t> o_wqkv(NL), o_wo(NL), o_wfc1(NL), o_wfc2(NL), o_bqkv(NL), o_bo(NL), o_bfc1(NL), o_bfc2(NL);
    for (int l = 0; l < NL; l++) {
        o_wqkv[l] = place((size_t)3 * D * D * es);
        o_wo[l] = place((size_t)D * D * es);
        o_wfc1[l] = place((size_t)c.mlp * D * es);
        o_wfc2[l] = place((size_t)D * c.mlp * es);
    }
    const size_t o_wout = place((size_t)M * D * es);
    const size_t o_bin = place((size_t)D * 4);
    for (int l = 0; l < NL; l++) {
        o_bqkv[l] = place((size_t)3 * D * 4);
        o_bo[l] = place((size_t)D * 4);
        o_bfc1[l] = place((size_t)c.mlp * 4);
        o_bfc2[l] = place((size_t)D * 4);
    }
    const size_t o_bout = place((size_t)M * 4);
    const size_t weights_end = off;
    const size_t o_mods = place((size_t)NS * NL * 6 * D * 4);
    const size_t o_fmods = place((size_t)NS * 2 * D * 4);
    const size_t o_t = place((size_t)(NS + 1) * 4);
    const size_t o_dt = place((size_t)NS * 4);
    const size_t o_temb = place((size_t)NS * D * 4);
    const size_t consts_end = off;
    const size_t o_hist = place((size_t)B * 8);
    const size_t o_pos = place((size_t)B * 8);
    const size_t o_plen = place((size_t)B * 4);
    const size_t o_keys = place((size_t)B * 8);
    const size_t o_spk = place((size_t)B * M * 4);
    const size_t o_carry = place((size_t)B * s->stream_stride * es);
    const size_t carry_end = off;
    const int rows_max = std::max(B * 2 * c.f_call, 2 * c.f_prompt);
    const int x_rows = std::max(B * c.f_call, c.f_prompt);
    const size_t q_elems = std::max((size_t)B * 2 * c.heads * round_up(c.f_call, 64) * 64,
                                    (size_t)2 * c.heads * round_up(c.f_prompt, 64) * 64);
    const size_t o_xin = place((size_t)rows_max * 4 * M * es);
    const size_t o_h = place((size_t)rows_max * D * 4);
    const size_t o_a = place((size_t)rows_max * D * es);
    const size_t o_o = place((size_t)rows_max * D * es);
    const size_t o_u = place((size_t)rows_max * c.mlp * es);
    const size_t o_q = place(q_elems * es);
    const size_t o_v = place((size_t)rows_max * M * 4);
    const size_t o_x = place((size_t)x_rows * M * 4);
    const size_t o_mu = place((size_t)x_rows * M * 4);
    const size_t o_mel = place((size_t)B * c.f_call * M * 4);
    const size_t o_cond = place((size_t)c.f_prompt * M * 4);
    const size_t o_gather = place((size_t)(c.f_retained + c.f_prompt) * D * 4);
    s->arena_bytes = off;

    hipError_t e = hipSuccess;
    if (c.hip_stream) {
        s->stream = (hipStream_t)c.hip_stream;
    } else {
        e = hipStreamCreateWithFlags(&s->stream, hipStreamNonBlocking);
        if (e != hipSuccess) {
            delete s;
            return fail(nullptr, DC_EDEVICE, std::string("dc_flow_init: ") + hipGetErrorString(e));
        }
        s->own_stream = true;
    }
    e = hipMalloc((void**)&s->arena, s->arena_bytes);
    if (e != hipSuccess) {
        s->arena = nullptr;
        dc_flow_free(s);
        return fail(nullptr, DC_ENOMEM, "dc_flow_init: device allocation of the arena failed");
    }
    char* A = s->arena;
    s->w_in = A + o_win;
    s->w_out = A + o_wout;
    s->b_in = (float*)(A + o_bin);
    s->b_out = (float*)(A + o_bout);
    for (int l = 0; l < NL; l++) {
        s->w_qkv.push_back(A + o_wqkv[l]);
        s->w_o.push_back(A + o_wo[l]);
        s->w_fc1.push_back(A + o_wfc1[l]);
        s->w_fc2.push_back(A + o_wfc2[l]);
        s->b_qkv.push_back((float*)(A + o_bqkv[l]));
        s->b_o.push_back((float*)(A + o_bo[l]));
        s->b_fc1.push_back((float*)(A + o_bfc1[l]));
        s->b_fc2.push_back((float*)(A + o_bfc2[l]));
    }
    s->mods = (float*)(A + o_mods);
    s->fmods = (float*)(A + o_fmods);
    s->t = (float*)(A + o_t);
    s->dt = (float*)(A + o_dt);
    s->silu_temb = (float*)(A + o_temb);
    s->hist = (int64_t*)(A + o_hist);
    s->pos = (int64_t*)(A + o_pos);
    s->plen = (int*)(A + o_plen);
    s->keys = (uint64_t*)(A + o_keys);
    s->spk = (float*)(A + o_spk);
    s->carry = A + o_carry;
    s->xin = A + o_xin;
    s->h = (float*)(A + o_h);
    s->a = A + o_a;
    s->o = A + o_o;
    s->u = A + o_u;
    s->q = A + o_q;
    s->v = (float*)(A + o_v);
    s->x = (float*)(A + o_x);
    s->mu_in = (float*)(A + o_mu);
    s->mel_out = (float*)(A + o_mel);
    s->cond_in = (float*)(A + o_cond);
    s->gather = (float*)(A + o_gather);

    // host image of the weight region: the per-step Linear weights in the
    // operand type (round to nearest even for bf16), biases in fp32
    std::vector<char> host(weights_end, 0);
    auto put_w = [&](size_t at, int64_t src, size_t n) {
        if (s->bf) {
            uint16_t* d = (uint16_t*)(host.data() + at);
            for (size_t i = 0; i < n; i++) {
                uint32_t u;
                std::memcpy(&u, blob + src + i, 4);
                if ((u & 0x7f800000u) == 0x7f800000u) d[i] = (uint16_t)((u >> 16) | ((u & 0x007fffffu) ? 0x40u : 0u));
                else d[i] = (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
            }
        } else {
            std::memcpy(host.data() + at, blob + src, n * 4);
        }
    };
    auto put_b = [&](size_t at, int64_t src, size_t n) { std::memcpy(host.data() + at, blob + src, n * 4); };
    put_w(o_win, bm.inW, (size_t)D * 4 * M);
    put_b(o_bin, bm.inb, D);
    for (int l = 0; l < NL; l++) {
        put_w(o_wqkv[l], bm.qkvW[l], (size_t)3 * D * D);
        put_b(o_bqkv[l], bm.qkvb[l], (size_t)3 * D);
        put_w(o_wo[l], bm.oW[l], (size_t)D * D);
        put_b(o_bo[l], bm.ob[l], D);
        put_w(o_wfc1[l], bm.fc1W[l], (size_t)c.mlp * D);
        put_b(o_bfc1[l], bm.fc1b[l], c.mlp);
        put_w(o_wfc2[l], bm.fc2W[l], (size_t)D * c.mlp);
        put_b(o_bfc2[l], bm.fc2b[l], D);
    }
    put_w(o_wout, bm.outW, (size_t)M * D);
    put_b(o_bout, bm.outb, M);
    e = hipMemcpy(A, host.data(), weights_end, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemsetAsync(A + weights_end, 0, s->arena_bytes - weights_end, s->stream);

    // per-step constants from the fp32 time MLP and ada layers, on the device
    // (a temporary copy of the blob, released once they are computed)
    float* tmp = nullptr;
    if (e == hipSuccess) e = hipMalloc((void**)&tmp, (size_t)bm.total * 4);
    if (e == hipSuccess) e = hipMemcpy(tmp, blob, (size_t)bm.total * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) {
        ConstParams cp{tmp + bm.t1W, tmp + bm.t1b, tmp + bm.t2W, tmp + bm.t2b, tmp + bm.ada[0], bm.block_stride,
                       tmp + bm.fadaW, s->silu_temb, s->mods, s->fmods, s->t, s->dt, NS, NL, D, c.t_dim};
        e = launch_consts(cp, s->stream);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (tmp) (void)hipFree(tmp);
    // warm-up: one direct call loads every code object; then the stream
    // state goes back to "no turn" (the carry's values are never read before
    // a prompt pass writes them) and stream b's noise key is set to b
    int count = 0;
    if (e == hipSuccess) e = enqueue_call(s, 0, B, c.f_call, 0, s->mu_in, nullptr, s->mel_out, s->stream, &count);
    if (e == hipSuccess) e = hipMemsetAsync(A + o_hist, 0, o_spk - o_hist, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e == hipSuccess) {
        std::vector<uint64_t> k(B);
        for (int b = 0; b < B; b++) k[b] = (uint64_t)b;
        e = hipMemcpy(s->keys, k.data(), (size_t)B * 8, hipMemcpyHostToDevice);
    }
    s->st.kernels_per_call = count;
    if (e == hipSuccess && !(c.flags & DC_NO_GRAPH)) {
        hipStream_t cs = nullptr;
        e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
        if (e == hipSuccess) {
            const hipError_t le = enqueue_call(s, 0, B, c.f_call, 0, s->mu_in, nullptr, s->mel_out, cs, nullptr);
            e = hipStreamEndCapture(cs, &s->graph);
            if (le != hipSuccess) e = le;
        }
        if (e == hipSuccess) e = hipGraphInstantiate(&s->exec, s->graph, nullptr, nullptr, 0);
        if (e == hipSuccess) {
            size_t nodes = 0;
            if (hipGraphGetNodes(s->graph, nullptr, &nodes) == hipSuccess) s->st.graph_nodes = (int32_t)nodes;
        }
        if (cs) (void)hipStreamDestroy(cs);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) {
        const std::string m = std::string("dc_flow_init: ") + hipGetErrorString(e);
        dc_flow_free(s);
        return fail(nullptr, DC_EDEVICE, m);
    }
    s->st.weight_bytes = (int64_t)consts_end;
    s->st.carry_bytes = (int64_t)(carry_end - o_carry);
    s->st.carry_live_bytes = (int64_t)B * NS * NL * 4 * (int64_t)(c.f_retained + c.f_prompt) * D * (int64_t)es;
    s->st.arena_bytes = (int64_t)s->arena_bytes;
    s->st.capture_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    *out = s;
    return DC_OK;
}

dc_status dc_flow_prompt(dc_flow_state* s, int32_t b, const float* mu, const float* cond, const float* spk,
                         int32_t frames)
{
    if (!s) return DC_EINVAL;
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned");
    const dc_flow_cfg& c = s->cfg;
    if (!mu || !cond || !spk) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "mu, cond or spk is NULL");
    }
    if (b < 0 || b >= c.batch || frames < 1 || frames > c.f_prompt) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "stream index or prompt length out of range");
    }
    const hipMemcpyKind k = (c.flags & DC_HOST_PTRS) ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice;
    const size_t fb = (size_t)frames * c.n_mel * 4;
    hipError_t e = hipMemcpyAsync(s->mu_in, mu, fb, k, s->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(s->cond_in, cond, fb, k, s->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(s->spk + (size_t)b * c.n_mel, spk, (size_t)c.n_mel * 4, k, s->stream);
    if (e == hipSuccess) e = launch_advance(s->hist, s->pos, s->plen, 0, b, frames, c.batch, c.f_chunk, s->stream);
    // the prompt frames' own solution is not an output
    if (e == hipSuccess) e = enqueue_call(s, b, 1, frames, 1, s->mu_in, s->cond_in, nullptr, s->stream, nullptr);
    if (e == hipSuccess) e = launch_advance(s->hist, s->pos, s->plen, 1, b, frames, c.batch, c.f_chunk, s->stream);
    if (e != hipSuccess) return device_fail(s, e, "prompt pass");
    s->plen_host[b] = frames;
    s->hist_host[b] = 0;
    s->st.prompts++;
    if (c.flags & DC_HOST_PTRS) return dc_flow_sync(s);
    return DC_OK;
}

dc_status dc_flow_decode_chunk(dc_flow_state* s, const float* mu, int32_t n, float* mel_out)
{
    if (!s) return DC_EINVAL;
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned");
    const dc_flow_cfg& c = s->cfg;
    if (!mu || !mel_out) {
        s->st.rejected++;
        return fail(s, DC_EINVAL, "mu or mel_out is NULL");
    }
    if (n < 1 || n > c.f_call) {
        s->st.rejected++;
        return fail(s, DC_ERANGE, "n must be in [1, f_call]");
    }
    for (int b = 0; b < c.batch; b++)
        if (s->plen_host[b] == 0) {
            s->st.rejected++;
            return fail(s, DC_ESTATE, "a stream has no turn: call dc_flow_prompt first");
        }
    const bool host = (c.flags & DC_HOST_PTRS) != 0;
    const size_t bytes = (size_t)c.batch * n * c.n_mel * 4;
    hipError_t e = hipSuccess;
    if (mu != s->mu_in) e = hipMemcpyAsync(s->mu_in, mu, bytes, host ? hipMemcpyHostToDevice : hipMemcpyDeviceToDevice, s->stream);
    if (e != hipSuccess) return device_fail(s, e, "mu staging");
    if (n == c.f_call && s->exec) {
        e = hipGraphLaunch(s->exec, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "hipGraphLaunch");
        s->st.replays++;
    } else {
        e = enqueue_call(s, 0, c.batch, n, 0, s->mu_in, nullptr, s->mel_out, s->stream, nullptr);
        if (e != hipSuccess) return device_fail(s, e, "direct launch");
        s->st.direct++;
    }
    s->st.calls++;
    host_advance(s, n);
    if (mel_out != s->mel_out) {
        e = hipMemcpyAsync(mel_out, s->mel_out, bytes, host ? hipMemcpyDeviceToHost : hipMemcpyDeviceToDevice, s->stream);
        if (e != hipSuccess) return device_fail(s, e, "mel staging");
    }
    if (host) return dc_flow_sync(s);
    return DC_OK;
}

dc_status dc_flow_sync(dc_flow_state* s)
{
    if (!s) return DC_EINVAL;
    const hipError_t e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "hipStreamSynchronize");
    return DC_OK;
}

dc_status dc_flow_carry_read(dc_flow_state* s, int32_t b, int32_t step, int32_t layer, int32_t branch, int32_t kv,
                             float* host_out, int32_t* frames)
{
    if (!s || !frames) return DC_EINVAL;
    const dc_flow_cfg& c = s->cfg;
    if (b < 0 || b >= c.batch || step < 0 || step >= c.n_steps || layer < 0 || layer >= c.depth || branch < 0 ||
        branch > 1 || kv < 0 || kv > 1)
        return fail(s, DC_EINVAL, "index out of range");
    const int64_t nh = std::min<int64_t>(s->hist_host[b], s->R);
    const int ext = s->plen_host[b] == 0 ? 0 : (int)(nh * c.f_chunk + s->plen_host[b]);
    *frames = ext;
    if (!host_out || ext == 0) return DC_OK;
    hipError_t e = launch_carry_gather(carry_ref(s, step, layer), b, branch, kv, c.heads, s->bf ? 1 : 0, ext,
                                       c.f_chunk, s->gather, s->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(host_out, s->gather, (size_t)ext * c.dim * 4, hipMemcpyDeviceToHost, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (e != hipSuccess) return device_fail(s, e, "carry read");
    return DC_OK;
}

dc_status dc_flow_profile(dc_flow_state* s, int32_t reps, dc_flow_kernel_stat* out, int32_t max, int32_t* count)
{
    if (!s || !count || reps < 1 || (out && max < 0)) return DC_EINVAL;
    if (s->poisoned) return fail(s, DC_ESTATE, "state is poisoned");
    const dc_flow_cfg& c = s->cfg;
    for (int b = 0; b < c.batch; b++)
        if (s->plen_host[b] == 0) return fail(s, DC_ESTATE, "a stream has no turn: call dc_flow_prompt first");
    const int nl = s->st.kernels_per_call;
    Recorder rec;
    rec.role.assign(nl, "");
    rec.flops.assign(nl, 0.0);
    rec.bytes.assign(nl, 0.0);
    rec.mfma.assign(nl, 0);
    rec.ev.assign(2 * (size_t)nl, nullptr);
    hipError_t e = hipSuccess;
    for (auto& ev : rec.ev)
        if (e == hipSuccess) e = hipEventCreate(&ev);
    std::vector<double> us(nl, 0.0);
    int launched = 0;
    for (int r = 0; r < reps && e == hipSuccess; r++) {
        rec.at = 0;
        e = enqueue_call(s, 0, c.batch, c.f_call, 0, s->mu_in, nullptr, s->mel_out, s->stream, &launched, &rec);
        if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
        for (size_t i = 0; i < rec.at && e == hipSuccess; i++) {
            float ms = 0.f;
            e = hipEventElapsedTime(&ms, rec.ev[2 * i], rec.ev[2 * i + 1]);
            us[i] += 1000.0 * ms / reps;
        }
    }
    for (auto& ev : rec.ev)
        if (ev) (void)hipEventDestroy(ev);
    if (e != hipSuccess) return device_fail(s, e, "profile");
    std::vector<dc_flow_kernel_stat> groups;
    for (size_t i = 0; i < rec.at; i++) {
        auto it = std::find_if(groups.begin(), groups.end(),
                               [&](const dc_flow_kernel_stat& g) { return rec.role[i] == g.name; });
        if (it == groups.end()) {
            dc_flow_kernel_stat g{};
            std::snprintf(g.name, sizeof(g.name), "%s", rec.role[i].c_str());
            g.mfma = rec.mfma[i];
            groups.push_back(g);
            it = groups.end() - 1;
        }
        it->launches++;
        it->us += us[i];
        it->flops += rec.flops[i];
        it->bytes += rec.bytes[i];
    }
    *count = (int32_t)groups.size();
    if (out)
        for (int i = 0; i < (int)groups.size() && i < max; i++) out[i] = groups[i];
    return DC_OK;
}

dc_status dc_flow_get_stats(const dc_flow_state* s, dc_flow_stats* out)
{
    if (!s || !out) return DC_EINVAL;
    *out = s->st;
    return DC_OK;
}

const char* dc_flow_last_error(const dc_flow_state* s) { return s ? s->msg.c_str() : g_flow_init_error.c_str(); }

void dc_flow_free(dc_flow_state* s)
{
    if (!s) return;
    if (s->stream) (void)hipStreamSynchronize(s->stream);
    if (s->exec) (void)hipGraphExecDestroy(s->exec);
    if (s->graph) (void)hipGraphDestroy(s->graph);
    if (s->arena) (void)hipFree(s->arena);
    if (s->own_stream && s->stream) (void)hipStreamDestroy(s->stream);
    delete s;
}

}  // extern "C"
