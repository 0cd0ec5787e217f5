// host_ffn.cpp -- the host tier: one token's expert FFN on host cores, reading the experts' blobs straight
// from the host store.  The paper's run recipe keeps the experts of some layers in host memory and computes
// them on the CPU (sec. 6, Fig. 3); here a residency rule picks which experts stay there (moe_cache_desc's
// host tier) and this file computes them while the GPU handles the rest.
//
// Plain host C++, built by the host compiler.  Work is split over a pool of threads in two phases: the
// gate/up row pairs of every expert (SwiGLU, combine weight folded in), then the output rows (each summed by
// one thread over the experts in rank order).  The dot products have AVX-512, AVX2 and portable forms, picked
// once from what the CPU supports.  x and the activations are stored twice: in order, and split into even and
// odd elements per block (32 elements for bf16, one 128-element group for int4) so that a vector load of
// packed weights meets the values it multiplies without shuffles.
#include <immintrin.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

#include "../../include/moe_budget.h"
#include "host_ffn.h"

namespace moe {
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();
}  // namespace moe

namespace {

enum Isa { kPortable = 0, kAvx2 = 1, kAvx512 = 2 };

Isa detect_isa() {
    __builtin_cpu_init();
    if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw")) return kAvx512;
    if (__builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma")) return kAvx2;
    return kPortable;
}

inline float bf16f(uint16_t b) {
    uint32_t u = uint32_t(b) << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

// A vector of K fp32 values in both orders (see the file comment).
struct Vec {
    const float *nat;  // [K] in order
    const float *ev;   // [K/2] even elements of each block
    const float *od;   // [K/2] odd elements of each block
};

// Block of the even/odd split: 32 elements for bf16 weights (one 64-byte load), 128 for int4 (one group).
inline int split_block(int dtype) { return dtype == MOE_INT4G128 ? 128 : 32; }

// Index of element i in the even (or odd) array.
inline size_t split_index(size_t i, int B) { return (i / B) * (B / 2) + (i % B) / 2; }

void split_store(float v, size_t i, int B, float *ev, float *od) {
    (i % 2 ? od : ev)[split_index(i, B)] = v;
}

// ---------------------------------------------------------------- dots ---
float dot_f32_portable(const float *w, const float *x, int K) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int i = 0; i < K; i += 8)
        for (int u = 0; u < 8; ++u) acc[u] += w[i + u] * x[i + u];
    return ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

__attribute__((target("avx2,fma"))) float dot_f32_avx2(const float *w, const float *x, int K) {
    __m256 a0 = _mm256_setzero_ps(), a1 = _mm256_setzero_ps();
    for (int i = 0; i < K; i += 16) {
        a0 = _mm256_fmadd_ps(_mm256_loadu_ps(w + i), _mm256_loadu_ps(x + i), a0);
        a1 = _mm256_fmadd_ps(_mm256_loadu_ps(w + i + 8), _mm256_loadu_ps(x + i + 8), a1);
    }
    alignas(32) float t[8];
    _mm256_store_ps(t, _mm256_add_ps(a0, a1));
    return ((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7]));
}

__attribute__((target("avx512f,avx512bw"))) float dot_f32_avx512(const float *w, const float *x, int K) {
    __m512 a0 = _mm512_setzero_ps(), a1 = _mm512_setzero_ps();
    for (int i = 0; i < K; i += 32) {
        a0 = _mm512_fmadd_ps(_mm512_loadu_ps(w + i), _mm512_loadu_ps(x + i), a0);
        a1 = _mm512_fmadd_ps(_mm512_loadu_ps(w + i + 16), _mm512_loadu_ps(x + i + 16), a1);
    }
    return _mm512_reduce_add_ps(_mm512_add_ps(a0, a1));
}

float dot_bf16_portable(const uint16_t *w, const Vec &x, int K) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int i = 0; i < K; i += 8)
        for (int u = 0; u < 8; ++u) acc[u] += bf16f(w[i + u]) * x.nat[i + u];
    return ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

// A 32-bit lane of packed bf16 holds element 2i in its low half and 2i + 1 in its high half: shifting left by
// 16 gives the even element as fp32, masking the low half gives the odd one.
__attribute__((target("avx2,fma"))) float dot_bf16_avx2(const uint16_t *w, const Vec &x, int K) {
    const __m256i hi_mask = _mm256_set1_epi32(int(0xffff0000u));
    __m256 a0 = _mm256_setzero_ps(), a1 = _mm256_setzero_ps();
    for (int i = 0; i < K; i += 16) {  // 16 elements: half of a 32-element block
        const __m256i v = _mm256_loadu_si256(reinterpret_cast<const __m256i *>(w + i));
        const size_t s = split_index(size_t(i), 32);
        a0 = _mm256_fmadd_ps(_mm256_castsi256_ps(_mm256_slli_epi32(v, 16)), _mm256_loadu_ps(x.ev + s), a0);
        a1 = _mm256_fmadd_ps(_mm256_castsi256_ps(_mm256_and_si256(v, hi_mask)), _mm256_loadu_ps(x.od + s), a1);
    }
    alignas(32) float t[8];
    _mm256_store_ps(t, _mm256_add_ps(a0, a1));
    return ((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7]));
}

__attribute__((target("avx512f,avx512bw"))) float dot_bf16_avx512(const uint16_t *w, const Vec &x, int K) {
    const __m512i hi_mask = _mm512_set1_epi32(int(0xffff0000u));
    __m512 a0 = _mm512_setzero_ps(), a1 = _mm512_setzero_ps(), a2 = _mm512_setzero_ps(), a3 = _mm512_setzero_ps();
    int i = 0;
    for (; i + 64 <= K; i += 64) {  // two 32-element blocks per pass
        const __m512i v0 = _mm512_loadu_si512(w + i), v1 = _mm512_loadu_si512(w + i + 32);
        const size_t s = size_t(i) / 2;
        a0 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(v0, 16)), _mm512_loadu_ps(x.ev + s), a0);
        a1 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_and_si512(v0, hi_mask)), _mm512_loadu_ps(x.od + s), a1);
        a2 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(v1, 16)), _mm512_loadu_ps(x.ev + s + 16), a2);
        a3 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_and_si512(v1, hi_mask)), _mm512_loadu_ps(x.od + s + 16), a3);
    }
    for (; i < K; i += 32) {
        const __m512i v = _mm512_loadu_si512(w + i);
        const size_t s = size_t(i) / 2;
        a0 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_slli_epi32(v, 16)), _mm512_loadu_ps(x.ev + s), a0);
        a1 = _mm512_fmadd_ps(_mm512_castsi512_ps(_mm512_and_si512(v, hi_mask)), _mm512_loadu_ps(x.od + s), a1);
    }
    return _mm512_reduce_add_ps(_mm512_add_ps(_mm512_add_ps(a0, a1), _mm512_add_ps(a2, a3)));
}

// int4 rows: K/2 packed bytes (low nibble = even element, two's complement) and K/128 bf16 scales.
float dot_int4_portable(const uint8_t *q, const uint16_t *sc, const Vec &x, int K) {
    float acc = 0.f;
    for (int g = 0; g < K / 128; ++g) {
        float part[4] = {0, 0, 0, 0};
        for (int b = 0; b < 64; ++b) {
            const int byte = q[64 * g + b];
            const int lo = ((byte & 15) ^ 8) - 8, hi = ((byte >> 4) ^ 8) - 8;
            part[b & 3] += float(lo) * x.nat[128 * g + 2 * b] + float(hi) * x.nat[128 * g + 2 * b + 1];
        }
        acc += bf16f(sc[g]) * ((part[0] + part[1]) + (part[2] + part[3]));
    }
    return acc;
}

__attribute__((target("avx2,fma"))) float dot_int4_avx2(const uint8_t *q, const uint16_t *sc, const Vec &x, int K) {
    const __m128i m15 = _mm_set1_epi8(15), m8 = _mm_set1_epi8(8);
    __m256 acc = _mm256_setzero_ps();
    for (int g = 0; g < K / 128; ++g) {
        __m256 p0 = _mm256_setzero_ps(), p1 = _mm256_setzero_ps();
        for (int b = 0; b < 64; b += 16) {  // 16 bytes: 16 even and 16 odd elements
            const __m128i v = _mm_loadu_si128(reinterpret_cast<const __m128i *>(q + 64 * g + b));
            const __m128i lo = _mm_sub_epi8(_mm_xor_si128(_mm_and_si128(v, m15), m8), m8);
            const __m128i hi = _mm_sub_epi8(_mm_xor_si128(_mm_and_si128(_mm_srli_epi16(v, 4), m15), m8), m8);
            const float *xe = x.ev + 64 * g + b, *xo = x.od + 64 * g + b;
            p0 = _mm256_fmadd_ps(_mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(lo)), _mm256_loadu_ps(xe), p0);
            p0 = _mm256_fmadd_ps(_mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(_mm_srli_si128(lo, 8))),
                                 _mm256_loadu_ps(xe + 8), p0);
            p1 = _mm256_fmadd_ps(_mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(hi)), _mm256_loadu_ps(xo), p1);
            p1 = _mm256_fmadd_ps(_mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(_mm_srli_si128(hi, 8))),
                                 _mm256_loadu_ps(xo + 8), p1);
        }
        acc = _mm256_fmadd_ps(_mm256_add_ps(p0, p1), _mm256_set1_ps(bf16f(sc[g])), acc);
    }
    alignas(32) float t[8];
    _mm256_store_ps(t, acc);
    return ((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7]));
}

__attribute__((target("avx512f,avx512bw"))) float dot_int4_avx512(const uint8_t *q, const uint16_t *sc, const Vec &x,
                                                                  int K) {
    const __m128i m15 = _mm_set1_epi8(15), m8 = _mm_set1_epi8(8);
    __m512 acc = _mm512_setzero_ps();
    for (int g = 0; g < K / 128; ++g) {
        __m512 p0 = _mm512_setzero_ps(), p1 = _mm512_setzero_ps();
        for (int b = 0; b < 64; b += 16) {
            const __m128i v = _mm_loadu_si128(reinterpret_cast<const __m128i *>(q + 64 * g + b));
            const __m128i lo = _mm_sub_epi8(_mm_xor_si128(_mm_and_si128(v, m15), m8), m8);
            const __m128i hi = _mm_sub_epi8(_mm_xor_si128(_mm_and_si128(_mm_srli_epi16(v, 4), m15), m8), m8);
            p0 = _mm512_fmadd_ps(_mm512_cvtepi32_ps(_mm512_cvtepi8_epi32(lo)), _mm512_loadu_ps(x.ev + 64 * g + b), p0);
            p1 = _mm512_fmadd_ps(_mm512_cvtepi32_ps(_mm512_cvtepi8_epi32(hi)), _mm512_loadu_ps(x.od + 64 * g + b), p1);
        }
        acc = _mm512_fmadd_ps(_mm512_add_ps(p0, p1), _mm512_set1_ps(bf16f(sc[g])), acc);
    }
    return _mm512_reduce_add_ps(acc);
}

// ------------------------------------------------------------- layout ---
size_t row_bytes(int dtype, int K) {
    return dtype == MOE_INT4G128 ? size_t(K) / 2 : size_t(K) * (dtype == MOE_F32 ? 4 : 2);
}

// Dot product of row r of one matrix of a blob.  `m` is the matrix's byte offset in the blob, R its rows.
float row_dot(Isa isa, int dtype, const uint8_t *blob, size_t m, int R, int r, int K, const Vec &x) {
    const uint8_t *row = blob + m + size_t(r) * row_bytes(dtype, K);
    if (dtype == MOE_F32) {
        const float *w = reinterpret_cast<const float *>(row);
        return isa == kAvx512 ? dot_f32_avx512(w, x.nat, K)
                              : isa == kAvx2 ? dot_f32_avx2(w, x.nat, K) : dot_f32_portable(w, x.nat, K);
    }
    if (dtype == MOE_BF16) {
        const uint16_t *w = reinterpret_cast<const uint16_t *>(row);
        return isa == kAvx512 ? dot_bf16_avx512(w, x, K)
                              : isa == kAvx2 ? dot_bf16_avx2(w, x, K) : dot_bf16_portable(w, x, K);
    }
    const uint16_t *sc = reinterpret_cast<const uint16_t *>(blob + m + size_t(R) * (K / 2)) + size_t(r) * (K / 128);
    return isa == kAvx512 ? dot_int4_avx512(row, sc, x, K)
                          : isa == kAvx2 ? dot_int4_avx2(row, sc, x, K) : dot_int4_portable(row, sc, x, K);
}

// Byte offset of W_d in a blob (W_gu [2I x H] first, int4 with its scales).
size_t down_offset(int H, int I, int dtype) {
    if (dtype == MOE_INT4G128) return size_t(I) * H + size_t(2) * I * (H / 128) * 2;
    return size_t(2) * I * H * (dtype == MOE_F32 ? 4 : 2);
}

}  // namespace

// ------------------------------------------------------------- the pool ---
struct moe_host_tier {
    int nt = 1;
    Isa isa = kPortable;
    std::vector<std::thread> workers;
    std::mutex mu;
    std::condition_variable cv;
    std::atomic<uint64_t> gen{0};
    std::atomic<int> pending{0};
    std::atomic<int> sleepers{0};
    std::atomic<bool> quit{false};
    bool busy = false;  // a call has begun and not yet finished
    // the current call
    const float *x = nullptr;
    int H = 0, I = 0, dtype = 0, n = 0;
    const uint8_t *blobs[MOE_MAX_TOPK] = {};
    float w[MOE_MAX_TOPK] = {};
    float *y = nullptr;
    std::vector<float> xs, acts;  // x split (even | odd); activations [n x I] in order, then split
    // work handed out in chunks: phase 1 (gate/up row pairs), then phase 2 (output rows) once phase 1 is done
    size_t n1 = 0, n2 = 0;  // chunks of each phase
    std::atomic<size_t> next1{0}, done1{0}, next2{0}, done2{0};
};

namespace {

// Idle threads spin this long before they sleep: long enough to bridge the gap between two layers' calls
// of a decode step, short enough not to hold the cores while the process does other work.
constexpr auto kSpinFor = std::chrono::milliseconds(2);

// Takes chunks until both phases are handed out: phase-1 chunks, then (once every phase-1 chunk is done,
// since each output row needs every activation) phase-2 chunks.  Each row is computed by whichever thread takes
// its chunk, with the same arithmetic, so the result does not depend on the schedule.
void gateup_chunk(moe_host_tier *t, size_t chunk);
void down_chunk(moe_host_tier *t, size_t chunk);

void work(moe_host_tier *t) {
    for (size_t c; (c = t->next1.fetch_add(1, std::memory_order_relaxed)) < t->n1;) {
        gateup_chunk(t, c);
        t->done1.fetch_add(1, std::memory_order_release);
    }
    while (t->done1.load(std::memory_order_acquire) < t->n1) _mm_pause();
    for (size_t c; (c = t->next2.fetch_add(1, std::memory_order_relaxed)) < t->n2;) {
        down_chunk(t, c);
        t->done2.fetch_add(1, std::memory_order_release);
    }
}

void worker(moe_host_tier *t) {
    uint64_t seen = 0;
    for (;;) {
        auto t0 = std::chrono::steady_clock::now();
        unsigned spins = 0;
        uint64_t g;
        while ((g = t->gen.load(std::memory_order_acquire)) == seen) {
            if (t->quit.load(std::memory_order_acquire)) return;
            _mm_pause();
            if ((++spins & 1023) == 0 && std::chrono::steady_clock::now() - t0 > kSpinFor) {
                std::unique_lock<std::mutex> lk(t->mu);
                t->sleepers.fetch_add(1);
                t->cv.wait(lk, [&] { return t->gen.load() != seen || t->quit.load(); });
                t->sleepers.fetch_sub(1);
                t0 = std::chrono::steady_clock::now();
            }
        }
        seen = g;
        if (t->quit.load(std::memory_order_acquire)) return;
        work(t);
        t->pending.fetch_sub(1, std::memory_order_acq_rel);
    }
}

// Row pairs (phase 1) and output rows (phase 2) per chunk: a few hundred KiB of weights each, so that the
// threads stay busy to the end however unevenly they start.
constexpr size_t kPairsPerChunk = 16, kRowsPerChunk = 32;

// Phase 1: act_j[i] = w_j * silu(W_g^j[i] . x) * (W_u^j[i] . x) for one chunk of the n*I pairs.
void gateup_chunk(moe_host_tier *t, size_t chunk) {
    const int H = t->H, I = t->I, dt = t->dtype, B = split_block(dt);
    const Vec x{t->x, t->xs.data(), t->xs.data() + H / 2};
    float *act = t->acts.data();
    float *aev = act + size_t(t->n) * I, *aod = aev + size_t(t->n) * I / 2;
    const size_t b = chunk * kPairsPerChunk, e = std::min(b + kPairsPerChunk, size_t(t->n) * I);
    for (size_t p = b; p < e; ++p) {
        const int j = int(p / size_t(I)), i = int(p % size_t(I));
        const float g = row_dot(t->isa, dt, t->blobs[j], 0, 2 * I, 2 * i, H, x);
        const float u = row_dot(t->isa, dt, t->blobs[j], 0, 2 * I, 2 * i + 1, H, x);
        const float a = t->w[j] * (g / (1.f + expf(-g)) * u);
        act[size_t(j) * I + i] = a;
        split_store(a, size_t(i), B, aev + size_t(j) * I / 2, aod + size_t(j) * I / 2);
    }
}

// Phase 2: y[h] = sum_j W_d^j[h] . act_j (rank order) for one chunk of the H rows.
void down_chunk(moe_host_tier *t, size_t chunk) {
    const int H = t->H, I = t->I, dt = t->dtype;
    const size_t doff = down_offset(H, I, dt);
    const float *act = t->acts.data();
    const float *aev = act + size_t(t->n) * I, *aod = aev + size_t(t->n) * I / 2;
    const size_t b = chunk * kRowsPerChunk, e = std::min(b + kRowsPerChunk, size_t(H));
    for (size_t h = b; h < e; ++h) {
        float acc = 0.f;
        for (int j = 0; j < t->n; ++j) {
            const Vec a{act + size_t(j) * I, aev + size_t(j) * I / 2, aod + size_t(j) * I / 2};
            acc += row_dot(t->isa, dt, t->blobs[j], doff, H, int(h), I, a);
        }
        t->y[h] = acc;
    }
}

}  // namespace

extern "C" {

int moe_host_tier_create(int threads, moe_host_tier **out) {
    if (!out) return moe::fail(MOE_ERR_INVALID_ARG, "host tier: NULL output");
    *out = nullptr;
    if (threads < 0 || threads > 1024) return moe::fail(MOE_ERR_INVALID_ARG, "host tier: threads %d outside [0, 1024]", threads);
    if (threads == 0) {
        cpu_set_t set;
        threads = sched_getaffinity(0, sizeof set, &set) == 0 ? CPU_COUNT(&set) : int(std::thread::hardware_concurrency());
        if (threads < 1) threads = 1;
    }
    auto *t = new moe_host_tier();
    t->nt = threads;
    t->isa = detect_isa();
    try {
        for (int i = 1; i < threads; ++i) t->workers.emplace_back(worker, t);
    } catch (...) {
        moe_host_tier_destroy(t);
        return moe::fail(MOE_ERR_INVALID_ARG, "host tier: could not start %d threads", threads);
    }
    *out = t;
    moe::clear_error();
    return MOE_OK;
}

int moe_host_tier_destroy(moe_host_tier *t) {
    if (!t) return MOE_OK;
    {
        std::lock_guard<std::mutex> lk(t->mu);
        t->quit.store(true);
    }
    t->cv.notify_all();
    for (auto &th : t->workers) th.join();
    delete t;
    return MOE_OK;
}

int moe_host_expert_ffn(moe_host_tier *t, const float *x, int H, int I, int w_dtype, int n, const void *const *blobs,
                        const float *weights, float *y_out) {
    int st = moe::host_ffn_begin(t, x, H, I, w_dtype, n, blobs, weights, y_out);
    return st == MOE_OK ? moe::host_ffn_finish(t) : st;
}

}  // extern "C"

namespace moe {

int host_ffn_begin(moe_host_tier *t, const float *x, int H, int I, int w_dtype, int n, const void *const *blobs,
                   const float *weights, float *y_out) {
    if (!t || !x || !y_out || (n > 0 && (!blobs || !weights)))
        return fail(MOE_ERR_INVALID_ARG, "host expert FFN: NULL argument");
    if (t->busy) return fail(MOE_ERR_INVALID_ARG, "host expert FFN: the tier is still working on a call");
    if (H <= 0 || I <= 0 || H % 128 || I % 128 || n < 0 || n > MOE_MAX_TOPK ||
        (w_dtype != MOE_F32 && w_dtype != MOE_BF16 && w_dtype != MOE_INT4G128))
        return fail(MOE_ERR_INVALID_ARG, "host expert FFN: unsupported H=%d I=%d n=%d dtype=%d", H, I, n, w_dtype);
    for (int j = 0; j < n; ++j)
        if (!blobs[j]) return fail(MOE_ERR_INVALID_ARG, "host expert FFN: blob %d is NULL", j);
    t->x = x;
    t->H = H;
    t->I = I;
    t->dtype = w_dtype;
    t->n = n;
    t->y = y_out;
    t->busy = true;
    if (n == 0) {
        t->n1 = t->n2 = 0;
        return MOE_OK;
    }
    for (int j = 0; j < n; ++j) {
        t->blobs[j] = static_cast<const uint8_t *>(blobs[j]);
        t->w[j] = weights[j];
    }
    const int B = split_block(w_dtype);
    t->xs.resize(size_t(H));
    for (int i = 0; i < H; ++i) split_store(x[i], size_t(i), B, t->xs.data(), t->xs.data() + H / 2);
    t->acts.resize(size_t(2) * n * I);
    t->n1 = (size_t(n) * I + kPairsPerChunk - 1) / kPairsPerChunk;
    t->n2 = (size_t(H) + kRowsPerChunk - 1) / kRowsPerChunk;
    t->next1.store(0, std::memory_order_relaxed);
    t->done1.store(0, std::memory_order_relaxed);
    t->next2.store(0, std::memory_order_relaxed);
    t->done2.store(0, std::memory_order_relaxed);
    t->pending.store(t->nt - 1, std::memory_order_relaxed);
    {
        std::lock_guard<std::mutex> lk(t->mu);
        t->gen.fetch_add(1, std::memory_order_acq_rel);  // releases the call's fields to the workers
    }
    if (t->sleepers.load() > 0) t->cv.notify_all();
    return MOE_OK;
}

int host_ffn_finish(moe_host_tier *t) {
    if (!t || !t->busy) return fail(MOE_ERR_INVALID_ARG, "host expert FFN: no call to finish");
    if (t->n == 0) {
        memset(t->y, 0, sizeof(float) * size_t(t->H));
    } else {
        work(t);  // the caller takes what is left
        while (t->done2.load(std::memory_order_acquire) < t->n2) _mm_pause();
        while (t->pending.load(std::memory_order_acquire) != 0) _mm_pause();  // every worker is out of the call
    }
    t->busy = false;
    clear_error();
    return MOE_OK;
}

}  // namespace moe
