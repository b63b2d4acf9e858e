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
// over host threads; the chunk partials of a (sequence, head) are merged by
// LSE at the end.  Vector code uses AVX-512 when the CPU has it (16 fp32 per
// instruction); otherwise (or with WSK_CPU_ENGINE=plain) plain loops compute
// the same quantities.
//
// Fused multiply-add contraction is off for the scalar code, which therefore
// follows the written order; the vector code uses explicit FMAs.
#pragma clang fp contract(off)

#include <immintrin.h>

#include <algorithm>
#include <atomic>
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

struct Job {
    const CpuAttendArgs *x;
    bool vec;
    std::vector<Item> items;
    std::vector<Partial> parts;   // one per item
};

// Rows of token t of KV head g (K row, V row).
inline void rows_of(const CpuAttendArgs &x, int i, int g, int t, const uint16_t *&k, const uint16_t *&v) {
    const int32_t slot = x.tables[i][t / x.block_tokens];
    const uint16_t *base = x.pool + (int64_t)slot * x.slot_elems;
    const int off = t % x.block_tokens;
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

// The AVX-512 path where the CPU has it, unless WSK_CPU_ENGINE=plain asks for
// the plain loops (which the tests also check on AVX-512 machines).
bool use_avx512() {
    static const bool ok = [] {
        const char *e = getenv("WSK_CPU_ENGINE");
        if (e && std::string(e) == "plain") return false;
        return __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw");
    }();
    return ok;
}

}  // namespace

int cpu_attend(const CpuAttendArgs &x) {
    Job job;
    job.x = &x;
    job.vec = use_avx512() && x.row_elems % 16 == 0 && x.dv % 16 == 0;
    const int hkv = x.mla ? 1 : x.n_q_heads / x.group;
    for (int i = 0; i < x.n; ++i)
        for (int g = 0; g < hkv; ++g)
            for (int a = x.start[i]; a < x.end[i]; a += kChunk) job.items.push_back({i, g, a, std::min(x.end[i], a + kChunk)});
    job.parts.resize(job.items.size());
    std::atomic<size_t> next{0};
    auto worker = [&]() {
        std::vector<float> qf;
        for (;;) {
            const size_t k = next.fetch_add(1);
            if (k >= job.items.size()) break;
            if (job.vec)
                run_item<true>(x, job.items[k], job.parts[k], qf);
            else
                run_item<false>(x, job.items[k], job.parts[k], qf);
        }
    };
    const int nth = std::max(1, std::min<int>(x.threads, (int)job.items.size()));
    std::vector<std::thread> pool;
    try {
        for (int t = 1; t < nth; ++t) pool.emplace_back(worker);
    } catch (...) {
        // fewer threads than asked: the ones that started and this one finish the work
    }
    worker();
    for (auto &th : pool) th.join();

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
