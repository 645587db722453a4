// Host-side driver of the C ABI for a sanitized build (AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code of the runtimes).  It walks
// dc_init and dc_flow_init over many valid and invalid configurations and
// every entry point's NULL-state path.  Without a GPU a valid configuration
// runs the whole host set-up (validation, network, tile choice, launch
// schedule, arena layout) and fails at the first device allocation; with one
// it initialises and frees the state.  Prints one line per failed expectation
// and exits non-zero if any failed.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "dc.h"
#include "dc_flow.h"

static int g_failures = 0;
static int g_calls = 0;

static void expect(bool ok, const char* what, int detail)
{
    if (!ok) {
        std::printf("FAILED: %s (%d)\n", what, detail);
        g_failures++;
    }
}

static dc_cfg tiny_cfg()
{
    dc_cfg c{};
    c.abi_version = DC_ABI_VERSION;
    c.vocab = 256, c.embed = 64, c.frames_per_token = 1;
    c.n_pre = 4, c.pre_kernel = 3;
    c.n_stages = 3;
    c.up_rate[0] = 2, c.up_rate[1] = 2, c.up_rate[2] = 4;
    c.channels[0] = 64, c.channels[1] = 32, c.channels[2] = 16, c.channels[3] = 8;
    c.n_rb = 1, c.rb_kernel[0] = 3;
    c.n_dil = 2, c.dil[0] = 1, c.dil[1] = 3;
    c.head_kernel = 7, c.n_fft = 16, c.hop = 4;
    c.lrelu_slope = 0.1f;
    c.dtype = DC_F32;
    c.batch = 1, c.chunk_tokens = 8, c.max_tokens = 8;
    c.sine_amp = 0.1f, c.noise_std = 0.003f, c.voiced_threshold = 10.0f, c.sample_rate = 24000.0f;
    return c;
}

static dc_cfg real_cfg()
{
    dc_cfg c = tiny_cfg();
    c.vocab = 6561, c.embed = 512, c.frames_per_token = 2;
    c.n_pre = 8;
    c.up_rate[0] = 8, c.up_rate[1] = 5, c.up_rate[2] = 3;
    c.channels[0] = 512, c.channels[1] = 256, c.channels[2] = 128, c.channels[3] = 64;
    c.n_rb = 3, c.rb_kernel[0] = 3, c.rb_kernel[1] = 7, c.rb_kernel[2] = 11;
    c.n_dil = 3, c.dil[0] = 1, c.dil[1] = 3, c.dil[2] = 5;
    c.chunk_tokens = 25, c.max_tokens = 25;
    return c;
}

// A valid configuration: initialises (and is freed) with a device, else fails
// at the first device allocation; the error text must be set either way.
static void valid(const dc_cfg& c, const char* what)
{
    const int64_t n = dc_blob_floats(&c);
    expect(n > 0, what, (int)n);
    std::vector<float> blob((size_t)(n > 0 ? n : 1), 0.0f);
    dc_state* s = reinterpret_cast<dc_state*>(&blob);   // must be overwritten
    const dc_status st = dc_init(blob.data(), (size_t)n * sizeof(float), &c, &s);
    g_calls++;
    if (st == DC_OK) {
        expect(s != nullptr, what, st);
        dc_stats stats{};
        expect(dc_get_stats(s, &stats) == DC_OK, what, 0);
        dc_free(s);
    } else {
        expect(st == DC_ENOMEM || st == DC_EDEVICE, what, st);
        expect(s == nullptr, what, st);
        const char* e = dc_last_error(nullptr);
        expect(e != nullptr && e[0] != 0, what, st);
    }
}

static void invalid(dc_cfg c, const char* what, dc_status want = DC_EINVAL)
{
    const int64_t n = dc_blob_floats(&c);
    std::vector<float> blob((size_t)(n > 0 ? n : 1), 0.0f);
    dc_state* s = nullptr;
    const dc_status st = dc_init(blob.data(), (size_t)(n > 0 ? n : 1) * sizeof(float), &c, &s);
    g_calls++;
    expect(st == want && s == nullptr, what, st);
}

static void vocoder()
{
    const dc_cfg base[2] = {tiny_cfg(), real_cfg()};
    for (int a = 0; a < 2; a++)
        for (int dt = 0; dt < 2; dt++)
            for (int batch : {1, 3, 8, 16, 128})
                for (int chunk : {1, 4, 25})
                    for (uint32_t flags : {0u, (uint32_t)DC_NO_FUSE, (uint32_t)DC_NO_RING,
                                           (uint32_t)(DC_NO_GRAPH | DC_HOST_PTRS)})
                        for (int nh : {0, 8}) {
                            dc_cfg c = base[a];
                            c.dtype = dt ? DC_BF16 : DC_F32;
                            c.batch = batch;
                            c.chunk_tokens = chunk;
                            c.max_tokens = 4 * chunk;
                            c.flags = flags;
                            c.n_harmonics = nh;
                            valid(c, "valid configuration");
                        }
    // every forced tile shape (1-based) on both architectures and dtypes
    for (int a = 0; a < 2; a++)
        for (int dt = 0; dt < 2; dt++)
            for (int v = 1; v <= 64; v++) {
                dc_cfg c = base[a];
                c.dtype = dt ? DC_BF16 : DC_F32;
                c.batch = dt ? 16 : 1;
                c.tile_variant = v;
                const int64_t n = dc_blob_floats(&c);
                std::vector<float> blob((size_t)n, 0.0f);
                dc_state* s = nullptr;
                const dc_status st = dc_init(blob.data(), (size_t)n * sizeof(float), &c, &s);
                g_calls++;
                // past the last shape: rejected before any device work
                expect(st == DC_OK || st == DC_ENOMEM || st == DC_EDEVICE || st == DC_EINVAL, "forced tile shape", v);
                if (st == DC_OK) dc_free(s);
            }

    dc_cfg c = real_cfg();
    invalid([&] { dc_cfg x = c; x.batch = 0; return x; }(), "batch 0");
    invalid([&] { dc_cfg x = c; x.chunk_tokens = 0; return x; }(), "chunk 0");
    invalid([&] { dc_cfg x = c; x.max_tokens = x.chunk_tokens - 1; return x; }(), "max below chunk");
    invalid([&] { dc_cfg x = c; x.n_stages = DC_MAX_STAGES + 1; return x; }(), "too many stages");
    invalid([&] { dc_cfg x = c; x.n_rb = DC_MAX_RB + 1; return x; }(), "too many branches");
    invalid([&] { dc_cfg x = c; x.n_dil = 0; return x; }(), "no dilations");
    invalid([&] { dc_cfg x = c; x.vocab = 0; return x; }(), "empty vocabulary");
    invalid([&] { dc_cfg x = c; x.dtype = 7; return x; }(), "unknown dtype");
    invalid([&] { dc_cfg x = c; x.tile_variant = -1; return x; }(), "negative tile shape");
    invalid([&] { dc_cfg x = c; x.n_harmonics = 99; return x; }(), "too many harmonics");
    invalid([&] { dc_cfg x = c; x.abi_version = DC_ABI_VERSION + 1; return x; }(), "abi version", DC_EVERSION);
    {
        const int64_t n = dc_blob_floats(&c);
        std::vector<float> blob((size_t)n + 1, 0.0f);
        dc_state* s = nullptr;
        expect(dc_init(blob.data(), (size_t)(n + 1) * sizeof(float), &c, &s) == DC_EINVAL && !s, "blob size", 0);
        expect(dc_init(nullptr, (size_t)n * sizeof(float), &c, &s) == DC_EINVAL, "NULL blob", 0);
        expect(dc_init(blob.data(), (size_t)n * sizeof(float), nullptr, &s) == DC_EINVAL, "NULL cfg", 0);
        expect(dc_init(blob.data(), (size_t)n * sizeof(float), &c, nullptr) == DC_EINVAL, "NULL out", 0);
        g_calls += 4;
    }
    // the NULL-state path of every entry point
    int32_t tok[4] = {0, 1, 2, 3};
    float pcm[4];
    dc_stats stats{};
    expect(dc_decode_chunk(nullptr, tok, 4, pcm) == DC_EINVAL, "decode NULL state", 0);
    expect(dc_decode_chunk_f0(nullptr, tok, pcm, 4, pcm) == DC_EINVAL, "decode_f0 NULL state", 0);
    expect(dc_decode_chunk_f0_static(nullptr, tok, pcm, 4, pcm) == DC_EINVAL, "static NULL state", 0);
    expect(dc_reset(nullptr) == DC_EINVAL, "reset NULL", 0);
    expect(dc_reset_stream(nullptr, 0) == DC_EINVAL, "reset_stream NULL", 0);
    expect(dc_sync(nullptr) == DC_EINVAL, "sync NULL", 0);
    expect(dc_get_stats(nullptr, &stats) == DC_EINVAL, "stats NULL", 0);
    expect(dc_token_buffer(nullptr) == nullptr && dc_audio_buffer(nullptr) == nullptr, "buffers NULL", 0);
    expect(dc_samples_per_token(nullptr) == 0 && dc_blob_floats(nullptr) == 0, "sizes NULL", 0);
    expect(dc_samples_per_token(&c) == 960, "samples per token", (int)dc_samples_per_token(&c));
    dc_free(nullptr);
}

static dc_flow_cfg flow_cfg(bool real)
{
    dc_flow_cfg c{};
    c.abi_version = DC_FLOW_ABI_VERSION;
    if (real) {
        c.n_mel = 80, c.dim = 512, c.heads = 8, c.depth = 16, c.mlp = 2048, c.t_dim = 256, c.n_steps = 10;
        c.f_prompt = 302, c.f_retained = 100, c.f_chunk = 50, c.f_call = 56;
    } else {
        c.n_mel = 16, c.dim = 128, c.heads = 2, c.depth = 2, c.mlp = 256, c.t_dim = 32, c.n_steps = 4;
        c.f_prompt = 24, c.f_retained = 16, c.f_chunk = 8, c.f_call = 10;
    }
    c.batch = 1;
    c.dtype = DC_F32;
    c.cfg_rate = 0.7f;
    c.temperature = 1.0f;
    return c;
}

static void flow()
{
    for (int real = 0; real < 2; real++)
        for (int dt = 0; dt < 2; dt++)
            for (int batch : {1, 2, 16, 128})
                for (uint32_t flags : {0u, (uint32_t)(DC_NO_GRAPH | DC_HOST_PTRS)}) {
                    dc_flow_cfg c = flow_cfg(real);
                    c.dtype = dt ? DC_BF16 : DC_F32;
                    c.batch = batch;
                    c.flags = flags;
                    const int64_t n = dc_flow_blob_floats(&c);
                    expect(n > 0, "flow blob size", (int)n);
                    std::vector<float> blob((size_t)(n > 0 ? n : 1), 0.0f);
                    dc_flow_state* s = nullptr;
                    const dc_status st = dc_flow_init(blob.data(), (size_t)n * sizeof(float), &c, &s);
                    g_calls++;
                    if (st == DC_OK)
                        dc_flow_free(s);
                    else
                        expect((st == DC_ENOMEM || st == DC_EDEVICE) && s == nullptr, "flow valid configuration", st);
                }
    dc_flow_cfg c = flow_cfg(true);
    const int64_t n = dc_flow_blob_floats(&c);
    std::vector<float> blob((size_t)n + 1, 0.0f);
    dc_flow_state* s = nullptr;
    auto bad = [&](dc_flow_cfg x, const char* what, dc_status want) {
        const int64_t m = dc_flow_blob_floats(&x);
        std::vector<float> b((size_t)(m > 0 ? m : 1), 0.0f);
        dc_flow_state* t = nullptr;
        const dc_status st = dc_flow_init(b.data(), (size_t)(m > 0 ? m : 1) * sizeof(float), &x, &t);
        g_calls++;
        expect(st == want && t == nullptr, what, st);
    };
    bad([&] { dc_flow_cfg x = c; x.batch = 0; return x; }(), "flow batch 0", DC_EINVAL);
    bad([&] { dc_flow_cfg x = c; x.heads = 3; return x; }(), "flow head width", DC_EINVAL);
    bad([&] { dc_flow_cfg x = c; x.f_call = x.f_chunk - 1; return x; }(), "flow call below chunk", DC_EINVAL);
    bad([&] { dc_flow_cfg x = c; x.f_retained = x.f_chunk + 1; return x; }(), "flow retained not a multiple", DC_EINVAL);
    bad([&] { dc_flow_cfg x = c; x.abi_version = 99; return x; }(), "flow abi version", DC_EVERSION);
    expect(dc_flow_init(blob.data(), (size_t)(n + 1) * sizeof(float), &c, &s) == DC_EINVAL && !s, "flow blob size", 0);
    expect(dc_flow_blob_floats(nullptr) == 0, "flow size NULL", 0);
    expect(dc_flow_sync(nullptr) == DC_EINVAL && dc_flow_decode_chunk(nullptr, nullptr, 1, nullptr) == DC_EINVAL, "flow NULL state", 0);
    dc_flow_free(nullptr);
}

int main()
{
    vocoder();
    flow();
    std::printf("calls %d failures %d\n", g_calls, g_failures);
    return g_failures ? 1 : 0;
}
