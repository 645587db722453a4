/*
 * Plain CPU oracle of the streaming Token2Wav decode step (fp64).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or constant with the
 * GPU library; the two meet only in the float32 weight blob and the token ids
 * (data), which the seeded generators produce.
 *
 * What it computes is the offline definition of the decoder, one stream at a
 * time, in the order the definition reads.  The paper's claim (Design,
 * "Strict trace equivalence", Definition 2, and the representation invariant
 * of the region contract) is that the carried, replayed streaming step
 * reproduces exactly this offline result, so the oracle holds no carry and no
 * chunking at all: a chunked run must equal one offline call.
 *
 * The paper prints no layer shapes.  The structure below is the causal
 * convolutional vocoder named by the decode step (token embedding repeated to
 * the frame clock, Design, region contract paragraph: 2 frames per token;
 * a causal Conv1d pre-stack; ConvTranspose1d upsampling stages each followed
 * by a multi-receptive-field residual block; a head conv to log-magnitude and
 * phase; an inverse STFT with overlap-add, whose window is one of the
 * device-resident constants of the region contract).  Readings where the
 * paper is silent:
 *   - every conv is causal: cross-correlation with (k-1)*d zeros on the left,
 *     values at negative time are zero, PyTorch weight layouts;
 *   - LeakyReLU(0.1) precedes every conv of a resblock, every upsampling conv
 *     and the head; the pre-stack is conv -> LeakyReLU;
 *   - the transposed conv (kernel 2u, stride u) keeps its first F*u outputs;
 *   - a resblock kernel k_j runs, per dilation d, the pair
 *     z <- z + conv_{k,1}(phi(conv_{k,d}(phi(z)))), and the stage output is
 *     the mean of the branch results summed left to right;
 *   - the head's first n_fft/2+1 channels are log-magnitudes, the rest phases
 *     in radians, magnitude = exp(log-magnitude) without clipping;
 *   - the inverse DFT is the real inverse DFT (imaginary parts of the DC and
 *     Nyquist bins are ignored), the window the periodic Hann window, frames
 *     are not centred, and the overlap-add is divided by the constant
 *     sum_m w^2[n - hop*m] (1.5 for n_fft = 16, hop = 4);
 *   - with bf16 parameters every parameter is rounded to bfloat16 (round to
 *     nearest even) and the arithmetic stays fp64;
 *   - optionally (n_harmonics > 0) a harmonic-plus-noise excitation source,
 *     the stochastic input of the paper's vocoder (Design, clause (iii)
 *     effect classification: the harmonic generator draws device randomness
 *     on every call; the adapter's device-resident constants include the
 *     sinusoid frequency table and the harmonic multiplier), enters the last
 *     upsampling stage: see oc_source below.
 */
#include <math.h>
#include <stdio.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int vocab, embed, frames_per_token;
    int n_pre, pre_kernel;
    int n_stages;
    int up_rate[8];
    int channels[9];
    int n_rb;
    int rb_kernel[8];
    int n_dil;
    int dil[8];
    int head_kernel, n_fft, hop;
    double slope;
    /* harmonic source (off when n_harmonics == 0) */
    int n_harmonics;
    double sine_amp, noise_std, voiced_threshold, sample_rate;
} oc_arch;

/* ---------------------------------------------------------------- helpers */

/* LeakyReLU: phi(v) = v for v >= 0, slope * v otherwise. */
static double phi(double v, double slope) { return v >= 0.0 ? v : slope * v; }

/* float32 -> bfloat16 -> float32, round to nearest, ties to even. */
float oc_round_bf16(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) {          /* inf / nan: truncate */
        if (u & 0x007fffffu) u |= 0x00400000u;        /* keep nan quiet */
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u = (u + 0x7fffu + lsb) & 0xffff0000u;
    }
    float y;
    memcpy(&y, &u, 4);
    return y;
}

int oc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------ the layers */

/*
 * Causal dilated Conv1d.
 *   out[t][o] = b[o] + sum_{j<k} sum_{i<Ci} W[o][i][j] * v[t-(k-1-j)*d][i]
 * with v at negative time equal to 0.  W has PyTorch layout [Co][Ci][k];
 * v and out are time-major [T][C].  The weight is re-laid out [Co][k][Ci] so
 * that the inner sum walks memory in order; the order of the terms is the
 * one written above (tap j outer, input channel i inner).
 */
void oc_cconv(int Ci, int Co, int k, int d, long T,
              const double* W, const double* b, const double* v, double* out)
{
    double* Wt = (double*)malloc(sizeof(double) * (size_t)Co * k * Ci);
    for (int o = 0; o < Co; o++)
        for (int i = 0; i < Ci; i++)
            for (int j = 0; j < k; j++)
                Wt[((size_t)o * k + j) * Ci + i] = W[((size_t)o * Ci + i) * k + j];
#pragma omp parallel for schedule(static)
    for (long t = 0; t < T; t++) {
        for (int o = 0; o < Co; o++) {
            double acc = 0.0;
            for (int j = 0; j < k; j++) {
                long ts = t - (long)(k - 1 - j) * d;
                if (ts < 0) continue;
                const double* w = Wt + ((size_t)o * k + j) * Ci;
                const double* x = v + (size_t)ts * Ci;
                for (int i = 0; i < Ci; i++) acc += w[i] * x[i];
            }
            out[(size_t)t * Co + o] = b[o] + acc;
        }
    }
    free(Wt);
}

/*
 * Causal ConvTranspose1d with kernel 2u and stride u, first F*u outputs kept.
 *   out[q*u + r][o] = b[o] + sum_{m in {0,1}} sum_i W[i][o][r + m*u] * v[q-m][i]
 * for q in [0, F), r in [0, u); v at negative time is 0.  W has PyTorch
 * layout [Ci][Co][2u].  This is every input frame q scattering its kernel
 * over outputs q*u .. q*u+2u-1, restricted to the outputs before F*u.
 */
void oc_convt(int Ci, int Co, int u, long F,
              const double* W, const double* b, const double* v, double* out)
{
#pragma omp parallel for schedule(static)
    for (long q = 0; q < F; q++) {
        for (int r = 0; r < u; r++) {
            for (int o = 0; o < Co; o++) {
                double acc = 0.0;
                for (int m = 0; m < 2; m++) {
                    long qs = q - m;
                    if (qs < 0) continue;
                    for (int i = 0; i < Ci; i++)
                        acc += W[((size_t)i * Co + o) * (2 * u) + r + m * u] * v[(size_t)qs * Ci + i];
                }
                out[((size_t)q * u + r) * Co + o] = b[o] + acc;
            }
        }
    }
}

/*
 * Real inverse DFT of length N from bins 0..N/2 (numpy irfft convention):
 *   x[n] = (1/N) [Re X0 + (-1)^n Re X_{N/2}
 *                 + 2 sum_{kk=1}^{N/2-1} (Re X_kk cos(2 pi kk n/N) - Im X_kk sin(2 pi kk n/N))]
 * The imaginary parts of bins 0 and N/2 do not enter.
 */
void oc_irfft(int N, const double* re, const double* im, double* x)
{
    int h = N / 2;
    for (int n = 0; n < N; n++) {
        double s = re[0] + ((n & 1) ? -re[h] : re[h]);
        for (int kk = 1; kk < h; kk++) {
            double a = 2.0 * M_PI * (double)kk * (double)n / (double)N;
            s += 2.0 * (re[kk] * cos(a) - im[kk] * sin(a));
        }
        x[n] = s / (double)N;
    }
}

/* Periodic Hann window: w[n] = 0.5 - 0.5 cos(2 pi n / N). */
double oc_hann(int N, int n) { return 0.5 - 0.5 * cos(2.0 * M_PI * (double)n / (double)N); }

/* The overlap-add normaliser sum_m w^2[n - hop*m], evaluated at n = N-1
 * (a sample every frame position covers once the stream is running). */
double oc_ola_norm(int N, int hop)
{
    double s = 0.0;
    for (int n = N - 1; n >= 0; n -= hop) s += oc_hann(N, n) * oc_hann(N, n);
    return s;
}

/*
 * Inverse STFT of M frames given log-magnitude and phase [M][N/2+1]:
 *   X_m[kk] = exp(logmag) (cos ph + i sin ph), v_m = irfft(X_m),
 *   acc[t]  = sum over frames m with 0 <= t - hop*m < N of w[t-hop*m] v_m[t-hop*m],
 *             added in ascending m,
 *   pcm[t]  = acc[t] / sum_m w^2,   t in [0, hop*M).
 * Samples at or after hop*M still miss later frames and are not emitted.
 */
void oc_istft(int N, int hop, long M, const double* logmag, const double* phase, double* pcm)
{
    int nb = N / 2 + 1;
    double norm = oc_ola_norm(N, hop);
    double* frames = (double*)malloc(sizeof(double) * (size_t)M * N);
#pragma omp parallel for schedule(static)
    for (long m = 0; m < M; m++) {
        double re[64], im[64], x[128];
        for (int kk = 0; kk < nb; kk++) {
            double mag = exp(logmag[(size_t)m * nb + kk]);
            double ph = phase[(size_t)m * nb + kk];
            re[kk] = mag * cos(ph);
            im[kk] = mag * sin(ph);
        }
        oc_irfft(N, re, im, x);
        for (int n = 0; n < N; n++) frames[(size_t)m * N + n] = oc_hann(N, n) * x[n];
    }
#pragma omp parallel for schedule(static)
    for (long t = 0; t < (long)hop * M; t++) {
        double acc = 0.0;
        long mlo = 0;                      /* smallest m with t - hop*m < N */
        if (t - N + 1 > 0) mlo = (t - N + 1 + hop - 1) / hop;
        long mhi = t / hop;                /* largest m with t - hop*m >= 0 */
        if (mhi > M - 1) mhi = M - 1;
        for (long m = mlo; m <= mhi; m++) acc += frames[(size_t)m * N + (t - hop * m)];
        pcm[t] = acc / norm;
    }
    free(frames);
}

/* ------------------------------------------------------ the source */

/*
 * Philox4x64-10, the counter-based generator of Salmon, Moraes, Dror and Shaw
 * ("Parallel random numbers: as easy as 1, 2, 3", SC 2011), written from its
 * published definition: ten rounds of
 *   (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))
 * with the key advanced by the Weyl constants (W0, W1) before every round but
 * the first.  The paper's engine admits the vocoder because its generator is
 * counter-based: what a kernel draws is a function of its counter, not of
 * hidden host state (Design, clause (iii)).
 */
static void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo)
{
    unsigned __int128 p = (unsigned __int128)a * b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void oc_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; r++) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        uint64_t hi0, lo0, hi1, lo1;
        mulhilo64(M0, c0, &hi0, &lo0);
        mulhilo64(M1, c2, &hi1, &lo1);
        uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* A 64-bit draw -> uniform in (0, 1): the top 53 bits, centred in their cell. */
double oc_u01(uint64_t x) { return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0); }

/* Box-Muller: two uniforms -> two independent standard normals. */
void oc_box_muller(double u0, double u1, double* g0, double* g1)
{
    double r = sqrt(-2.0 * log(u0));
    *g0 = r * cos(2.0 * M_PI * u1);
    *g1 = r * sin(2.0 * M_PI * u1);
}

/*
 * Harmonic-plus-noise excitation of one stream (neural source filter of the
 * vocoder's harmonic generator; a reading of the paper, which names the
 * generator and its device-resident sinusoid frequency table and harmonic
 * multiplier but prints no formula):
 *   f0[f] >= 0 Hz per frame f of the pre-stack clock, S = prod(up_rate) * hop
 *   samples per frame, sample t = f*S + r.
 *   Sinusoid h = 0..H (multiplier h+1): increment inc_h[f] = (h+1) f0[f] / sr
 *   cycles per sample; phase at the start of frame f
 *     P_h[0] = phi_h,  P_h[f+1] = frac(P_h[f] + S * inc_h[f])   (frame order),
 *   phi_0 = 0 and phi_h = u01(Philox(ctr = (0, h, 1, 0))[0]) for h >= 1; the
 *   phase of sample t is frac(P_h[f] + (r+1) inc_h[f]) (the running sum
 *   includes sample t).
 *   Voiced frame: f0[f] > voiced_threshold.  e_h[t] = voiced * A sin(2 pi phase)
 *   + noise_h[t] * (voiced ? noise_std : A/3).
 *   Noise: Philox(key = (seed, stream), ctr = (t, g, 0, 0)) for group
 *   g = 0, 1, ..: its four draws give, by Box-Muller on (u0, u1) and (u2, u3),
 *   noise_{4g}, noise_{4g+1}, noise_{4g+2}, noise_{4g+3}.
 *   src[t] = tanh(mb + sum_{h=0..H} mw[h] e_h[t])  (h ascending).
 * Counters are sample indices since the stream's start, so a chunked decode
 * draws what an offline one does.  src receives F * S samples.
 */
void oc_source(const oc_arch* a, const double* f0, long F, uint64_t seed, uint64_t stream,
               const double* mw, double mb, double* src)
{
    int H1 = a->n_harmonics + 1;
    long S = a->hop;
    for (int s = 0; s < a->n_stages; s++) S *= a->up_rate[s];
    uint64_t key[2] = {seed, stream};
    double* P = (double*)malloc(sizeof(double) * (size_t)(F + 1) * H1);
    for (int h = 0; h < H1; h++) {
        double p0 = 0.0;
        if (h > 0) {
            uint64_t ctr[4] = {0, (uint64_t)h, 1, 0}, o[4];
            oc_philox4x64(ctr, key, o);
            p0 = oc_u01(o[0]);
        }
        P[h] = p0;
        for (long f = 0; f < F; f++) {
            double inc = (double)(h + 1) * f0[f] / a->sample_rate;
            double x = P[(size_t)f * H1 + h] + (double)S * inc;
            P[(size_t)(f + 1) * H1 + h] = x - floor(x);
        }
    }
    int groups = (H1 + 3) / 4;
#pragma omp parallel for schedule(static)
    for (long t = 0; t < F * S; t++) {
        long f = t / S, r = t - f * S;
        int voiced = f0[f] > a->voiced_threshold;
        double noise[64];
        for (int g = 0; g < groups; g++) {
            uint64_t ctr[4] = {(uint64_t)t, (uint64_t)g, 0, 0}, o[4];
            oc_philox4x64(ctr, key, o);
            oc_box_muller(oc_u01(o[0]), oc_u01(o[1]), &noise[4 * g], &noise[4 * g + 1]);
            oc_box_muller(oc_u01(o[2]), oc_u01(o[3]), &noise[4 * g + 2], &noise[4 * g + 3]);
        }
        double acc = 0.0;
        for (int h = 0; h < H1; h++) {
            double inc = (double)(h + 1) * f0[f] / a->sample_rate;
            double x = P[(size_t)f * H1 + h] + (double)(r + 1) * inc;
            double ph = x - floor(x);
            double e = (voiced ? a->sine_amp * sin(2.0 * M_PI * ph) : 0.0) +
                       noise[h] * (voiced ? a->noise_std : a->sine_amp / 3.0);
            acc += mw[h] * e;
        }
        src[t] = tanh(mb + acc);
    }
    free(P);
}

/* ---------------------------------------------------------- the decoder */

typedef struct {
    const float* p;
    int bf16;
} blob_reader;

/* Next tensor of the blob as fp64 (rounded to bf16 first if asked). */
static double* take(blob_reader* r, size_t n)
{
    double* out = (double*)malloc(sizeof(double) * n);
    for (size_t i = 0; i < n; i++) out[i] = r->bf16 ? (double)oc_round_bf16(r->p[i]) : (double)r->p[i];
    r->p += n;
    return out;
}

long oc_blob_floats(const oc_arch* a)
{
    long n = (long)a->vocab * a->embed;
    long c0 = a->channels[0];
    n += (long)a->n_pre * (c0 * c0 * a->pre_kernel + c0);
    for (int s = 0; s < a->n_stages; s++) {
        long ci = a->channels[s], co = a->channels[s + 1];
        n += ci * co * 2 * a->up_rate[s] + co;
        for (int j = 0; j < a->n_rb; j++) n += (long)a->n_dil * 2 * (co * co * a->rb_kernel[j] + co);
    }
    long hc = 2 * (a->n_fft / 2 + 1);
    n += hc * a->channels[a->n_stages] * a->head_kernel + hc;
    if (a->n_harmonics > 0) n += (a->n_harmonics + 1) + 1 + (long)a->channels[a->n_stages] * a->hop + a->channels[a->n_stages];
    return n;
}

long oc_samples_per_token(const oc_arch* a)
{
    long u = 1;
    for (int s = 0; s < a->n_stages; s++) u *= a->up_rate[s];
    return (long)a->frames_per_token * u * a->hop;
}

static void copy_tap(const char* want, const char* have, const double* x, size_t n, double* tap_out, int* found)
{
    if (want && tap_out && strcmp(want, have) == 0) {
        memcpy(tap_out, x, sizeof(double) * n);
        *found = 1;
    }
}

static double* phi_copy(const double* x, size_t n, double slope)
{
    double* y = (double*)malloc(sizeof(double) * n);
    for (size_t i = 0; i < n; i++) y[i] = phi(x[i], slope);
    return y;
}

/*
 * Offline decode of one stream of T tokens from the zero state.
 * pcm receives T * samples_per_token samples.  With the harmonic source,
 * f0 holds T * frames_per_token frame values (Hz) and (seed, stream) key its
 * generator; otherwise f0 may be NULL.  If tap_name names an intermediate
 * ("embed", "pre<l>", "s<s>.y", "s<s>.rb<j>.h<i>", "s<s>.rb<j>.z<i>",
 * "s<s>.x", "head", "src" -- the source samples as [frames of the last
 * stage][hop]) its [frames][C] values are copied to tap_out.  Returns 0 on
 * success, -1 on a bad argument, -2 if the tap name was given but never
 * produced.
 */
int oc_decode(const oc_arch* a, int bf16_params, const float* blob, long blob_n,
              const int32_t* ids, long T, const double* f0, uint64_t seed, uint64_t stream,
              double* pcm, const char* tap_name, double* tap_out)
{
    if (blob_n != oc_blob_floats(a) || T <= 0) return -1;
    if (a->n_harmonics > 0 && !f0) return -1;
    for (long t = 0; t < T; t++)
        if (ids[t] < 0 || ids[t] >= a->vocab) return -1;
    blob_reader rd = {blob, bf16_params};
    int found = 0;
    double slope = a->slope;

    /* token embedding, each token repeated frames_per_token times */
    int C = a->channels[0];
    long F = T * a->frames_per_token;
    double* emb = take(&rd, (size_t)a->vocab * a->embed);
    double* x = (double*)malloc(sizeof(double) * (size_t)F * C);
    for (long f = 0; f < F; f++) {
        long tok = ids[f / a->frames_per_token];
        memcpy(x + (size_t)f * C, emb + (size_t)tok * C, sizeof(double) * C);
    }
    free(emb);
    copy_tap(tap_name, "embed", x, (size_t)F * C, tap_out, &found);

    /* pre-stack: x <- phi(conv_{k,1}(x)) */
    char name[64];
    for (int l = 0; l < a->n_pre; l++) {
        int k = a->pre_kernel;
        double* W = take(&rd, (size_t)C * C * k);
        double* b = take(&rd, (size_t)C);
        double* y = (double*)malloc(sizeof(double) * (size_t)F * C);
        oc_cconv(C, C, k, 1, F, W, b, x, y);
        for (size_t i = 0; i < (size_t)F * C; i++) y[i] = phi(y[i], slope);
        free(W); free(b); free(x);
        x = y;
        snprintf(name, sizeof name, "pre%d", l);
        copy_tap(tap_name, name, x, (size_t)F * C, tap_out, &found);
    }

    /* upsampling stages, each followed by the multi-receptive-field block */
    for (int s = 0; s < a->n_stages; s++) {
        int ci = a->channels[s], co = a->channels[s + 1], u = a->up_rate[s];
        double* W = take(&rd, (size_t)ci * co * 2 * u);
        double* b = take(&rd, (size_t)co);
        double* xa = phi_copy(x, (size_t)F * ci, slope);
        long Fo = F * u;
        double* y = (double*)malloc(sizeof(double) * (size_t)Fo * co);
        oc_convt(ci, co, u, F, W, b, xa, y);
        free(W); free(b); free(xa); free(x);
        if (a->n_harmonics > 0 && s == a->n_stages - 1) {
            /* the source enters the last stage after its ConvTranspose1d:
             * y[tau][c] += bd[c] + sum_{j<hop} Wd[c][0][j] * src[tau*hop + j]
             * (a Conv1d from one channel, kernel = stride = hop) */
            blob_reader sr = {blob + (blob_n - ((a->n_harmonics + 1) + 1 + (long)co * a->hop + co)), bf16_params};
            double* mw = take(&sr, (size_t)a->n_harmonics + 1);
            double* mb = take(&sr, 1);
            double* Wd = take(&sr, (size_t)co * a->hop);
            double* bd = take(&sr, (size_t)co);
            long F0 = T * a->frames_per_token;
            double* src = (double*)malloc(sizeof(double) * (size_t)Fo * a->hop);
            oc_source(a, f0, F0, seed, stream, mw, mb[0], src);
            copy_tap(tap_name, "src", src, (size_t)Fo * a->hop, tap_out, &found);
            for (long t = 0; t < Fo; t++)
                for (int o = 0; o < co; o++) {
                    double sd = bd[o];
                    for (int j = 0; j < a->hop; j++) sd += Wd[(size_t)o * a->hop + j] * src[(size_t)t * a->hop + j];
                    y[(size_t)t * co + o] = y[(size_t)t * co + o] + sd;
                }
            free(mw); free(mb); free(Wd); free(bd); free(src);
        }
        snprintf(name, sizeof name, "s%d.y", s);
        copy_tap(tap_name, name, y, (size_t)Fo * co, tap_out, &found);

        size_t n = (size_t)Fo * co;
        double* sum = (double*)calloc(n, sizeof(double));
        double* z = (double*)malloc(sizeof(double) * n);
        double* h = (double*)malloc(sizeof(double) * n);
        double* c = (double*)malloc(sizeof(double) * n);
        for (int j = 0; j < a->n_rb; j++) {
            int k = a->rb_kernel[j];
            memcpy(z, y, sizeof(double) * n);
            for (int i = 0; i < a->n_dil; i++) {
                double* W1 = take(&rd, (size_t)co * co * k);
                double* b1 = take(&rd, (size_t)co);
                double* W2 = take(&rd, (size_t)co * co * k);
                double* b2 = take(&rd, (size_t)co);
                double* za = phi_copy(z, n, slope);
                oc_cconv(co, co, k, a->dil[i], Fo, W1, b1, za, h);
                snprintf(name, sizeof name, "s%d.rb%d.h%d", s, j, i);
                copy_tap(tap_name, name, h, n, tap_out, &found);
                double* ha = phi_copy(h, n, slope);
                oc_cconv(co, co, k, 1, Fo, W2, b2, ha, c);
                for (size_t e = 0; e < n; e++) z[e] = z[e] + c[e];
                snprintf(name, sizeof name, "s%d.rb%d.z%d", s, j, i);
                copy_tap(tap_name, name, z, n, tap_out, &found);
                free(za); free(ha); free(W1); free(b1); free(W2); free(b2);
            }
            for (size_t e = 0; e < n; e++) sum[e] = sum[e] + z[e];
        }
        for (size_t e = 0; e < n; e++) sum[e] = sum[e] / (double)a->n_rb;
        free(z); free(h); free(c); free(y);
        x = sum;
        F = Fo;
        C = co;
        snprintf(name, sizeof name, "s%d.x", s);
        copy_tap(tap_name, name, x, (size_t)F * C, tap_out, &found);
    }

    /* head conv -> log-magnitude | phase -> inverse STFT */
    int nb = a->n_fft / 2 + 1, hc = 2 * nb;
    double* Wh = take(&rd, (size_t)hc * C * a->head_kernel);
    double* bh = take(&rd, (size_t)hc);
    double* xa = phi_copy(x, (size_t)F * C, slope);
    double* sh = (double*)malloc(sizeof(double) * (size_t)F * hc);
    oc_cconv(C, hc, a->head_kernel, 1, F, Wh, bh, xa, sh);
    free(Wh); free(bh); free(xa); free(x);
    copy_tap(tap_name, "head", sh, (size_t)F * hc, tap_out, &found);
    double* lm = (double*)malloc(sizeof(double) * (size_t)F * nb);
    double* ph = (double*)malloc(sizeof(double) * (size_t)F * nb);
    for (long f = 0; f < F; f++)
        for (int kk = 0; kk < nb; kk++) {
            lm[(size_t)f * nb + kk] = sh[(size_t)f * hc + kk];
            ph[(size_t)f * nb + kk] = sh[(size_t)f * hc + nb + kk];
        }
    oc_istft(a->n_fft, a->hop, F, lm, ph, pcm);
    free(lm); free(ph); free(sh);
    long tail = a->n_harmonics > 0 ? (a->n_harmonics + 1) + 1 + (long)C * a->hop + C : 0;
    if (rd.p != blob + blob_n - tail) return -1;
    if (tap_name && tap_out && !found) return -2;
    return 0;
}
