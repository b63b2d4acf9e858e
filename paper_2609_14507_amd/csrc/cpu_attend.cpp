// In-place CPU attention over the CPU partition (the CPU engine of Sec. 5.1
// and Sec. 6.1): every query head attends a range of positions of its
// sequence, reading K/V (or MLA latent) rows where they sit in the host pool,
// block by block through the sequence's CPU block table, with no copy or
// reorganisation (Sec. 4.3 (iii)).  The output is the same normalised partial
// and natural-log LSE as the GPU's, ready for the LSE merge.
//
// Arithmetic: bf16 rows widened to fp32, fp32 dot products and accumulation,
// an online softmax over tiles of 16 tokens (one rescale per tile).  Work is
// cut into (sequence, KV head, chunk of at most kChunk tokens) items spread
// over a persistent pool of host threads; the chunk partials of a (sequence, head) are merged by
// LSE at the end.  Vector code uses AVX-512 (with bf16 dot products where the
// CPU has them); otherwise (or with WSK_CPU_ENGINE=plain / avx512) simpler
// loops compute the same quantities.
//
// Fused multiply-add contraction is off for the scalar code, which therefore
// follows the written order; the vector code uses explicit FMAs.
#pragma clang fp contract(off)

#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <memory>
#include <cmath>
#include <cstdlib>
#include <string>
#include <thread>
#include <vector>

#include "wsk.h"
#include "wsk_internal.h"

namespace wsk {
namespace {

constexpr int kChunk = 2048;   // tokens per work item
constexpr int kTok = 16;       // tokens per softmax tile

inline float bf16f(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    __builtin_memcpy(&f, &u, 4);
    return f;
}

struct Item {
    int i, g;          // sequence index, KV head
    int a, b;          // token range
};

struct Partial {       // per (item, head): running max (log2 domain), sum, unnormalised O
    std::vector<float> m, l, acc;
};

// ---- vector helpers -------------------------------------------------------
__attribute__((target("avx512f,avx512bw"))) inline __m512 load_bf16x16(const uint16_t *p) {
    const __m256i h = _mm256_loadu_si256((const __m256i *)p);
    return _mm512_castsi512_ps(_mm512_slli_epi32(_mm512_cvtepu16_epi32(h), 16));
}

// dot(q (fp32, n), row (bf16, n)), n % 16 == 0
__attribute__((target("avx512f,avx512bw"))) inline float dot512(const float *q, const uint16_t *row, int n) {
    __m512 s0 = _mm512_setzero_ps(), s1 = _mm512_setzero_ps();
    int d = 0;
    for (; d + 32 <= n; d += 32) {
        s0 = _mm512_fmadd_ps(_mm512_loadu_ps(q + d), load_bf16x16(row + d), s0);
        s1 = _mm512_fmadd_ps(_mm512_loadu_ps(q + d + 16), load_bf16x16(row + d + 16), s1);
    }
    for (; d < n; d += 16) s0 = _mm512_fmadd_ps(_mm512_loadu_ps(q + d), load_bf16x16(row + d), s0);
    return _mm512_reduce_add_ps(_mm512_add_ps(s0, s1));
}

// acc[0..n) += p * row[0..n)  (row bf16), n % 16 == 0
__attribute__((target("avx512f,avx512bw"))) inline void axpy512(float *acc, float p, const uint16_t *row, int n) {
    const __m512 pv = _mm512_set1_ps(p);
    for (int d = 0; d < n; d += 16)
        _mm512_storeu_ps(acc + d, _mm512_fmadd_ps(pv, load_bf16x16(row + d), _mm512_loadu_ps(acc + d)));
}

__attribute__((target("avx512f"))) inline void scale512(float *acc, float a, int n) {
    const __m512 av = _mm512_set1_ps(a);
    for (int d = 0; d < n; d += 16) _mm512_storeu_ps(acc + d, _mm512_mul_ps(av, _mm512_loadu_ps(acc + d)));
}

inline float dot_plain(const float *q, const uint16_t *row, int n) {
    float s = 0.f;
    for (int d = 0; d < n; ++d) s += q[d] * bf16f(row[d]);
    return s;
}
inline void axpy_plain(float *acc, float p, const uint16_t *row, int n) {
    for (int d = 0; d < n; ++d) acc[d] += p * bf16f(row[d]);
}
inline void scale_plain(float *acc, float a, int n) {
    for (int d = 0; d < n; ++d) acc[d] *= a;
}

enum class Path;

struct Job {
    const CpuAttendArgs *x;
    Path path;
    std::vector<Item> items;
    std::vector<Partial> parts;   // one per item
};

// Rows of token t of KV head g (K row, V row); block_tokens is a power of two.
inline void rows_of(const CpuAttendArgs &x, int i, int g, int t, const uint16_t *&k, const uint16_t *&v) {
    const int bshift = __builtin_ctz((unsigned)x.block_tokens);
    const int32_t slot = x.tables[i][t >> bshift];
    const uint16_t *base = x.pool + (int64_t)slot * x.slot_elems;
    const int off = t & (x.block_tokens - 1);
    if (x.mla) {
        k = base + (int64_t)off * x.row_elems;
        v = k;
    } else {
        const uint16_t *head = base + (int64_t)g * 2 * x.block_tokens * x.row_elems;
        k = head + (int64_t)off * x.row_elems;
        v = head + (int64_t)(x.block_tokens + off) * x.row_elems;
    }
}

template <bool kVec>
void run_item(const CpuAttendArgs &x, const Item &it, Partial &pt, std::vector<float> &qf) {
    const int G = x.group, dk = x.row_elems, dv = x.dv;
    const int h0 = it.g * G;
    // the item's query heads, widened to fp32
    qf.resize((size_t)G * dk);
    for (int h = 0; h < G; ++h)
        for (int d = 0; d < dk; ++d) qf[(size_t)h * dk + d] = bf16f(x.q[(int64_t)it.i * x.q_row + (int64_t)(h0 + h) * dk + d]);
    pt.m.assign(G, -INFINITY);
    pt.l.assign(G, 0.f);
    pt.acc.assign((size_t)G * dv, 0.f);
    float s[kTok];
    const uint16_t *krow[kTok], *vrow[kTok];
    for (int t0 = it.a; t0 < it.b; t0 += kTok) {
        const int nt = std::min(kTok, it.b - t0);
        for (int t = 0; t < nt; ++t) rows_of(x, it.i, it.g, t0 + t, krow[t], vrow[t]);
        for (int h = 0; h < G; ++h) {
            const float *qh = &qf[(size_t)h * dk];
            float mt = -INFINITY;
            for (int t = 0; t < nt; ++t) {
                s[t] = (kVec ? dot512(qh, krow[t], dk) : dot_plain(qh, krow[t], dk)) * x.scale_log2;
                mt = std::max(mt, s[t]);
            }
            const float m_new = std::max(pt.m[h], mt);
            float *acc = &pt.acc[(size_t)h * dv];
            if (m_new != pt.m[h]) {
                const float alpha = std::exp2(pt.m[h] - m_new);   // 0 for the first tile
                pt.l[h] *= alpha;
                if (kVec)
                    scale512(acc, alpha, dv);
                else
                    scale_plain(acc, alpha, dv);
                pt.m[h] = m_new;
            }
            for (int t = 0; t < nt; ++t) {
                const float p = std::exp2(s[t] - m_new);
                pt.l[h] += p;
                if (kVec)
                    axpy512(acc, p, vrow[t], dv);
                else
                    axpy_plain(acc, p, vrow[t], dv);
            }
        }
    }
}

// ---- AVX-512 with bf16 dot products ----------------------------------------
// A 16-token tile of K is transposed once into dim pairs x tokens, so that
// vdpbf16ps accumulates the 16 tokens' scores of one head in the 16 lanes of
// one register (products of bf16 values are exact in fp32; sums are fp32).
// exp2 over the 16 scores is vectorised: x = n + f with n the nearest integer
// and |f| <= 1/2, 2^f = e^(f ln 2) from the Taylor series of e^y to the y^7
// term (remainder below 6e-9 relative for |y| <= ln(2)/2), scaled by 2^n;
// results below 2^-126 (weights negligible next to the running maximum's 1)
// are 0.
// P.V keeps the accumulators of all heads for a block of columns in
// registers while the tile's V rows stream through.
constexpr int kMaxPairs = 288;   // 576 / 2

struct ScratchBf16 {
    alignas(64) uint32_t kt[kMaxPairs][16];   // K tile, dim pair j of token t at kt[j][t]
    alignas(64) float p[16][16];              // probabilities [head][token] (up to 16 heads)
    float alpha[16];
};

__attribute__((target("avx512f,avx512bw,avx512bf16"))) inline __m512 exp2v(__m512 x) {
    // below 2^-126 the result is 0 (no denormal probabilities); -inf -> 0
    const __mmask16 keep = _mm512_cmp_ps_mask(x, _mm512_set1_ps(-126.f), _CMP_GE_OQ);
    x = _mm512_max_ps(x, _mm512_set1_ps(-127.f));
    const __m512 n = _mm512_roundscale_ps(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
    const __m512 y = _mm512_mul_ps(_mm512_sub_ps(x, n), _mm512_set1_ps(0.69314718055994530942f));
    // 1 + y (1 + y/2 (1 + y/3 (1 + y/4 (1 + y/5 (1 + y/6 (1 + y/7))))))
    __m512 r = _mm512_fmadd_ps(y, _mm512_set1_ps(1.f / 7.f), _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(_mm512_mul_ps(y, _mm512_set1_ps(1.f / 6.f)), r, _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(_mm512_mul_ps(y, _mm512_set1_ps(1.f / 5.f)), r, _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(_mm512_mul_ps(y, _mm512_set1_ps(1.f / 4.f)), r, _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(_mm512_mul_ps(y, _mm512_set1_ps(1.f / 3.f)), r, _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(_mm512_mul_ps(y, _mm512_set1_ps(0.5f)), r, _mm512_set1_ps(1.f));
    r = _mm512_fmadd_ps(y, r, _mm512_set1_ps(1.f));
    return _mm512_maskz_scalef_ps(keep, r, n);
}

// max / sum over the 16 lanes, in every lane
__attribute__((target("avx512f,avx512bw,avx512bf16"))) inline __m512 allmax(__m512 v) {
    v = _mm512_max_ps(v, _mm512_shuffle_f32x4(v, v, 0x4e));
    v = _mm512_max_ps(v, _mm512_shuffle_f32x4(v, v, 0xb1));
    v = _mm512_max_ps(v, _mm512_permute_ps(v, 0x4e));
    return _mm512_max_ps(v, _mm512_permute_ps(v, 0xb1));
}
__attribute__((target("avx512f,avx512bw,avx512bf16"))) inline __m512 allsum(__m512 v) {
    v = _mm512_add_ps(v, _mm512_shuffle_f32x4(v, v, 0x4e));
    v = _mm512_add_ps(v, _mm512_shuffle_f32x4(v, v, 0xb1));
    v = _mm512_add_ps(v, _mm512_permute_ps(v, 0x4e));
    return _mm512_add_ps(v, _mm512_permute_ps(v, 0xb1));
}

// 16 x 16 transpose of 32-bit elements: out[j] holds element j of every in[t]
__attribute__((target("avx512f,avx512bw,avx512bf16"))) inline void transpose16(__m512i (&r)[16]) {
    __m512i t[16];
    for (int i = 0; i < 16; i += 2) {
        t[i] = _mm512_unpacklo_epi32(r[i], r[i + 1]);
        t[i + 1] = _mm512_unpackhi_epi32(r[i], r[i + 1]);
    }
    for (int i = 0; i < 16; i += 4) {
        r[i] = _mm512_unpacklo_epi64(t[i], t[i + 2]);
        r[i + 1] = _mm512_unpackhi_epi64(t[i], t[i + 2]);
        r[i + 2] = _mm512_unpacklo_epi64(t[i + 1], t[i + 3]);
        r[i + 3] = _mm512_unpackhi_epi64(t[i + 1], t[i + 3]);
    }
    // each 128-bit lane q of r[4b + c] now holds element 4q' + ... : finish with 128-bit shuffles
    for (int i = 0; i < 4; ++i) {
        t[i] = _mm512_shuffle_i32x4(r[i], r[i + 4], 0x88);
        t[i + 4] = _mm512_shuffle_i32x4(r[i], r[i + 4], 0xdd);
        t[i + 8] = _mm512_shuffle_i32x4(r[i + 8], r[i + 12], 0x88);
        t[i + 12] = _mm512_shuffle_i32x4(r[i + 8], r[i + 12], 0xdd);
    }
    for (int i = 0; i < 4; ++i) {
        r[i] = _mm512_shuffle_i32x4(t[i], t[i + 8], 0x88);
        r[i + 8] = _mm512_shuffle_i32x4(t[i], t[i + 8], 0xdd);
        r[i + 4] = _mm512_shuffle_i32x4(t[i + 4], t[i + 12], 0x88);
        r[i + 12] = _mm512_shuffle_i32x4(t[i + 4], t[i + 12], 0xdd);
    }
}

template <int G>
__attribute__((target("avx512f,avx512bw,avx512bf16"))) void run_item_bf16(const CpuAttendArgs &x, const Item &it,
                                                                          Partial &pt, std::vector<float> &qf,
                                                                          ScratchBf16 &sc) {
    const int dk = x.row_elems, dv = x.dv, npair = dk / 2;
    const int h0 = it.g * G;
    static const uint16_t zero_row[576] = {};
    // query pairs as raw bf16 bits (qf holds them as 32-bit words)
    qf.resize((size_t)G * npair);
    uint32_t *qp = reinterpret_cast<uint32_t *>(qf.data());
    for (int h = 0; h < G; ++h)
        __builtin_memcpy(qp + (size_t)h * npair, x.q + (int64_t)it.i * x.q_row + (int64_t)(h0 + h) * dk, dk * 2);
    pt.m.assign(G, -INFINITY);
    pt.l.assign(G, 0.f);
    pt.acc.assign((size_t)G * dv, 0.f);
    const uint16_t *krow[16], *vrow[16];
    const __m512 scale = _mm512_set1_ps(x.scale_log2);
    for (int t0 = it.a; t0 < it.b; t0 += 16) {
        const int nt = std::min(16, it.b - t0);
        for (int t = 0; t < 16; ++t) {
            if (t < nt)
                rows_of(x, it.i, it.g, t0 + t, krow[t], vrow[t]);
            else
                krow[t] = vrow[t] = zero_row;
        }
        // prefetch: the next tile's rows into L1 and the rows one block ahead
        // into L2.  A KV head's rows come in runs of one block a slot apart,
        // which the hardware prefetchers pick up late; the L2 stream keeps
        // the L1 prefetches short (measured on MI355X servers' EPYC hosts: 15.0 ->
        // 17.0 GB/s on one thread, +3-20 % on 16, against L1 only)
        {
            const int tq = t0 + 16;
            const int nq = std::min(16, it.b - tq);
            for (int t = 0; t < nq; ++t) {
                const uint16_t *pk, *pv;
                rows_of(x, it.i, it.g, tq + t, pk, pv);
                for (int off = 0; off < dk * 2; off += 64) _mm_prefetch((const char *)pk + off, _MM_HINT_T0);
                if (!x.mla)
                    for (int off = 0; off < dv * 2; off += 64) _mm_prefetch((const char *)pv + off, _MM_HINT_T0);
            }
        }
        {
            const int tp = t0 + x.block_tokens;
            const int np = std::min(16, it.b - tp);
            for (int t = 0; t < np; ++t) {
                const uint16_t *pk, *pv;
                rows_of(x, it.i, it.g, tp + t, pk, pv);
                for (int off = 0; off < dk * 2; off += 64) _mm_prefetch((const char *)pk + off, _MM_HINT_T1);
                if (!x.mla)
                    for (int off = 0; off < dv * 2; off += 64) _mm_prefetch((const char *)pv + off, _MM_HINT_T1);
            }
        }
        // K tile -> dim pairs x tokens
        for (int jb = 0; jb < npair; jb += 16) {
            __m512i r[16];
            for (int t = 0; t < 16; ++t) r[t] = _mm512_loadu_si512((const void *)(krow[t] + 2 * jb));
            transpose16(r);
            for (int j = 0; j < 16; ++j) _mm512_store_si512((void *)sc.kt[jb + j], r[j]);
        }
        const __mmask16 valid = (__mmask16)((1u << nt) - 1u);
        bool rescale = false;
        // scores of all G heads at once: one K pair row feeds G independent chains
        __m512 sacc[G];
        for (int h = 0; h < G; ++h) sacc[h] = _mm512_setzero_ps();
        for (int j = 0; j < npair; ++j) {
            const __m512bh kv = (__m512bh)_mm512_load_si512((const void *)sc.kt[j]);
            for (int h = 0; h < G; ++h)
                sacc[h] = _mm512_dpbf16_ps(sacc[h], kv, (__m512bh)_mm512_set1_epi32((int)qp[(size_t)h * npair + j]));
        }
        // online softmax, all in vector registers (max, sum and both exp2 over
        // broadcast lanes: no scalar round trip, no library call)
        for (int h = 0; h < G; ++h) {
            __m512 sv = _mm512_mul_ps(sacc[h], scale);
            sv = _mm512_mask_blend_ps(valid, _mm512_set1_ps(-INFINITY), sv);
            const __m512 mo = _mm512_set1_ps(pt.m[h]);
            const __m512 mn = _mm512_max_ps(mo, allmax(sv));
            const __m512 al = exp2v(_mm512_sub_ps(mo, mn));   // 0 for the first tile
            const __m512 pv = exp2v(_mm512_sub_ps(sv, mn));
            const float alpha = _mm512_cvtss_f32(al);
            sc.alpha[h] = alpha;
            rescale |= alpha != 1.f;
            pt.l[h] = pt.l[h] * alpha + _mm512_cvtss_f32(allsum(pv));
            pt.m[h] = _mm512_cvtss_f32(mn);
            _mm512_storeu_ps(sc.p[h], pv);
        }
        // O[h][cols] = alpha_h O[h][cols] + sum_t p[h][t] v_t[cols], columns in blocks of 16 x (16 / G)
        constexpr int cb = G <= 8 ? 32 : 16;   // columns per block: registers hold G x cb / 16 accumulators
        for (int c0 = 0; c0 < dv; c0 += cb) {
            __m512 acc[G][cb / 16];
            for (int h = 0; h < G; ++h)
                for (int u = 0; u < cb / 16; ++u) {
                    acc[h][u] = _mm512_loadu_ps(&pt.acc[(size_t)h * dv + c0 + 16 * u]);
                    if (rescale) acc[h][u] = _mm512_mul_ps(acc[h][u], _mm512_set1_ps(sc.alpha[h]));
                }
            for (int t = 0; t < nt; ++t)
                for (int u = 0; u < cb / 16; ++u) {
                    const __m512 v = load_bf16x16(vrow[t] + c0 + 16 * u);
                    for (int h = 0; h < G; ++h) acc[h][u] = _mm512_fmadd_ps(_mm512_set1_ps(sc.p[h][t]), v, acc[h][u]);
                }
            for (int h = 0; h < G; ++h)
                for (int u = 0; u < cb / 16; ++u) _mm512_storeu_ps(&pt.acc[(size_t)h * dv + c0 + 16 * u], acc[h][u]);
        }
    }
}

enum class Path { Plain, Avx512, Avx512Bf16 };

// The fastest path the CPU has; WSK_CPU_ENGINE=plain or =avx512 asks for a
// slower one (the tests check every path on a CPU that has them all).
Path cpu_path() {
    static const Path path = [] {
        const char *e = getenv("WSK_CPU_ENGINE");
        const bool f = __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw");
        const bool bf = f && __builtin_cpu_supports("avx512bf16");
        if (e && std::string(e) == "plain") return Path::Plain;
        if (e && std::string(e) == "avx512") return f ? Path::Avx512 : Path::Plain;
        return bf ? Path::Avx512Bf16 : f ? Path::Avx512 : Path::Plain;
    }();
    return path;
}

// Persistent host workers: a call wakes as many as it needs and works
// alongside them, so a call costs no thread creation.  Calls are serialised.
// The pool lives until the process ends (its threads block on a condition
// variable when idle).
class WorkerPool {
public:
    static WorkerPool &get() {
        static WorkerPool *pool = new WorkerPool;   // never destroyed: idle threads end with the process
        return *pool;
    }
    // runs f on the calling thread and on n_extra pool threads; returns when all are done
    void run(int n_extra, const std::function<void()> &f) {
        std::lock_guard<std::mutex> call(call_mu_);
        std::unique_lock<std::mutex> lk(mu_);
        try {
            while ((int)workers_.size() < n_extra) {
                const int idx = (int)workers_.size();
                workers_.emplace_back([this, idx] { loop(idx); });
            }
        } catch (...) {
            n_extra = (int)workers_.size();   // fewer threads: the rest of the work is shared by those
        }
        job_ = &f;
        want_ = n_extra;
        running_ = n_extra;
        ++epoch_;
        lk.unlock();
        wake_.notify_all();
        f();
        lk.lock();
        finished_.wait(lk, [&] { return running_ == 0; });
        job_ = nullptr;
    }

private:
    void loop(int idx) {
        uint64_t seen = 0;
        std::unique_lock<std::mutex> lk(mu_);
        for (;;) {
            wake_.wait(lk, [&] { return epoch_ != seen; });
            seen = epoch_;
            if (idx >= want_) continue;
            const std::function<void()> *f = job_;
            lk.unlock();
            (*f)();
            lk.lock();
            if (--running_ == 0) finished_.notify_all();
        }
    }
    std::mutex call_mu_, mu_;
    std::condition_variable wake_, finished_;
    std::vector<std::thread> workers_;
    const std::function<void()> *job_ = nullptr;
    uint64_t epoch_ = 0;
    int want_ = 0, running_ = 0;
};

}  // namespace

namespace {
// XOR of the 64-bit words of [p, p + n), read with 64-byte vector loads where
// the CPU has them.
__attribute__((target("avx512f"))) uint64_t fold_avx512(const uint64_t *p, size_t n) {
    __m512i a0 = _mm512_setzero_si512(), a1 = a0, a2 = a0, a3 = a0;
    size_t i = 0;
    for (; i + 32 <= n; i += 32) {
        a0 = _mm512_xor_si512(a0, _mm512_loadu_si512(p + i));
        a1 = _mm512_xor_si512(a1, _mm512_loadu_si512(p + i + 8));
        a2 = _mm512_xor_si512(a2, _mm512_loadu_si512(p + i + 16));
        a3 = _mm512_xor_si512(a3, _mm512_loadu_si512(p + i + 24));
    }
    alignas(64) uint64_t t[8];
    _mm512_store_si512(t, _mm512_xor_si512(_mm512_xor_si512(a0, a1), _mm512_xor_si512(a2, a3)));
    uint64_t r = 0;
    for (int k = 0; k < 8; ++k) r ^= t[k];
    for (; i < n; ++i) r ^= p[i];
    return r;
}
uint64_t fold_plain(const uint64_t *p, size_t n) {
    uint64_t r = 0;
    for (size_t i = 0; i < n; ++i) r ^= p[i];
    return r;
}
}  // namespace

uint64_t host_read(const void *p, size_t bytes, int threads) {
    const size_t piece = 4u << 20;   // 4 MiB per task
    const size_t n = (bytes + piece - 1) / piece;
    std::vector<uint64_t> part(n, 0);
    const bool vec = __builtin_cpu_supports("avx512f");
    parallel_tasks((int)n, threads, [&](int t) {
        const size_t a = (size_t)t * piece, len = std::min(piece, bytes - a) / 8;
        const uint64_t *w = reinterpret_cast<const uint64_t *>((const char *)p + a);
        part[t] = vec ? fold_avx512(w, len) : fold_plain(w, len);
    });
    uint64_t r = 0;
    for (uint64_t x : part) r ^= x;
    return r;
}

void parallel_tasks(int n_tasks, int threads, const std::function<void(int)> &task) {
    if (n_tasks <= 0) return;
    std::atomic<int> next{0};
    const std::function<void()> worker = [&]() {
        for (int k; (k = next.fetch_add(1)) < n_tasks;) task(k);
    };
    WorkerPool::get().run(std::max(0, std::min(threads, n_tasks) - 1), worker);
}

int cpu_attend(const CpuAttendArgs &x) {
    Job job;
    job.x = &x;
    const Path path = cpu_path();
    const bool shapes16 = x.row_elems % 32 == 0 && x.dv % 32 == 0 && x.row_elems <= 2 * kMaxPairs &&
                          (x.group == 1 || x.group == 2 || x.group == 4 || x.group == 8 || x.group == 16);
    job.path = path == Path::Avx512Bf16 && !shapes16 ? Path::Avx512 : path;
    if (job.path == Path::Avx512 && (x.row_elems % 16 || x.dv % 16)) job.path = Path::Plain;
    const int hkv = x.mla ? 1 : x.n_q_heads / x.group;
    for (int i = 0; i < x.n; ++i)
        for (int g = 0; g < hkv; ++g)
            for (int j = x.rbegin ? x.rbegin[i] : i; j < (x.rbegin ? x.rbegin[i + 1] : i + 1); ++j)
                for (int a = x.start[j]; a < x.end[j]; a += kChunk)
                    job.items.push_back({i, g, a, std::min(x.end[j], a + kChunk)});
    job.parts.resize(job.items.size());
    std::atomic<size_t> next{0};
    auto worker = [&]() {
        std::vector<float> qf;
        std::unique_ptr<ScratchBf16> sc(job.path == Path::Avx512Bf16 ? new ScratchBf16 : nullptr);
        for (;;) {
            const size_t k = next.fetch_add(1);
            if (k >= job.items.size()) break;
            if (job.path == Path::Avx512Bf16) {
                switch (x.group) {
                    case 1: run_item_bf16<1>(x, job.items[k], job.parts[k], qf, *sc); break;
                    case 2: run_item_bf16<2>(x, job.items[k], job.parts[k], qf, *sc); break;
                    case 4: run_item_bf16<4>(x, job.items[k], job.parts[k], qf, *sc); break;
                    case 8: run_item_bf16<8>(x, job.items[k], job.parts[k], qf, *sc); break;
                    default: run_item_bf16<16>(x, job.items[k], job.parts[k], qf, *sc); break;
                }
            }
            else if (job.path == Path::Avx512)
                run_item<true>(x, job.items[k], job.parts[k], qf);
            else
                run_item<false>(x, job.items[k], job.parts[k], qf);
        }
    };
    const int nth = std::max(1, std::min<int>(x.threads, (int)job.items.size()));
    WorkerPool::get().run(nth - 1, worker);

    // merge the chunk partials of every (sequence, head), in chunk order
    const int H = x.n_q_heads, G = x.group, dv = x.dv;
    std::vector<float> M((size_t)x.n * H, -INFINITY);
    for (size_t k = 0; k < job.items.size(); ++k) {
        const Item &it = job.items[k];
        for (int h = 0; h < G; ++h) {
            float &mm = M[(size_t)it.i * H + it.g * G + h];
            mm = std::max(mm, job.parts[k].m[h]);
        }
    }
    std::vector<double> L((size_t)x.n * H, 0.0);
    std::fill(x.o, x.o + (size_t)x.n * H * dv, 0.f);
    for (size_t k = 0; k < job.items.size(); ++k) {
        const Item &it = job.items[k];
        for (int h = 0; h < G; ++h) {
            const size_t row = (size_t)it.i * H + it.g * G + h;
            const float w = std::exp2(job.parts[k].m[h] - M[row]);
            L[row] += (double)w * job.parts[k].l[h];
            float *o = x.o + row * dv;
            const float *a = &job.parts[k].acc[(size_t)h * dv];
            for (int d = 0; d < dv; ++d) o[d] += w * a[d];
        }
    }
    for (size_t row = 0; row < (size_t)x.n * H; ++row) {
        float *o = x.o + row * dv;
        if (M[row] == -INFINITY) {   // empty range
            x.lse[row] = -INFINITY;
            continue;
        }
        const float inv = (float)(1.0 / L[row]);
        for (int d = 0; d < dv; ++d) o[d] *= inv;
        x.lse[row] = (float)((M[row] + std::log2(L[row])) * 0.69314718055994530942);
    }
    return 0;
}

}  // namespace wsk
