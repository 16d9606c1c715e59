// Table-lookup CPU kernel for the quantised widely-linear layer with int8
// activations (Sec. 3.4, the CPU-inference paragraph): four 2-bit codes form
// one 8-bit index, the partial sums of every index with the activations are
// tabulated once per token, and the row loop reduces to table fetches and
// integer adds.  The result is exact: the int32 sums equal the products of
// the ternary code planes of Eq. (realify-ops) with the int8 activations.
//
// Host code only (x86-64, SSE2).  One call processes one layer for B tokens;
// the work is spread over a persistent pool of host threads.
//
// Table: for token b and column group g (columns 4g .. 4g+3), entry
// lut[g][idx][b] holds four int16 sums over the group's columns m:
//   (sum b_re q_re, sum b_re q_im, sum b_im q_re, sum b_im q_im)
// with code (idx >> 2m) & 3 for column 4g+m, b_re + i b_im = i^code.  In the
// canonical packed layout four consecutive codes of a row are one byte, bits
// 2m for column 4g+m, so a code byte is the table index as stored.
//
// Loop: rows are taken in chunks of kRowChunk by the pool's threads; for each
// chunk the K range is walked in windows whose slice of the table fits the
// core's L2 cache, and inside a window all 2T planes (U and W, every stage)
// of a row fetch from the same table rows.  int16 partial sums are widened to
// int32 every kFlushGroups groups (|entry| <= 4 * 128, so 63 groups cannot
// overflow int16).

#include <emmintrin.h>
#include <sched.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "fairy2i.h"

namespace {

constexpr int kFlushGroups = 32;
constexpr int kRowChunk = 32;
constexpr int kMaxThreads = 256;
constexpr size_t kWindowBytes = 256 << 10;  // table slice per K window

// ---------------------------------------------------------------------------
// Persistent worker pool: run(n, f) calls f(w) for w = 0 .. n-1, worker 0 on
// the calling thread, and returns when all have finished.  Calls are
// serialised by a mutex.
// ---------------------------------------------------------------------------
class Pool {
 public:
  void run(int n, const std::function<void(int)>& f) {
    std::lock_guard<std::mutex> call_lock(call_mu_);
    resize(n);
    {
      std::lock_guard<std::mutex> l(mu_);
      job_ = &f;
      pending_ = n - 1;
      ++generation_;
    }
    cv_.notify_all();
    f(0);
    std::unique_lock<std::mutex> l(mu_);
    done_cv_.wait(l, [&] { return pending_ == 0; });
    job_ = nullptr;
  }

  ~Pool() { stop(); }

 private:
  void resize(int n) {
    if (static_cast<int>(workers_.size()) == n - 1) return;
    stop();
    stopping_ = false;
    // a new worker starts from the current generation, so it waits for the
    // next job even if it first runs after run() has published it
    const uint64_t gen = generation_;
    for (int w = 1; w < n; ++w) workers_.emplace_back([this, w, gen] { loop(w, gen); });
  }

  void stop() {
    {
      std::lock_guard<std::mutex> l(mu_);
      stopping_ = true;
      ++generation_;
    }
    cv_.notify_all();
    for (auto& t : workers_) t.join();
    workers_.clear();
  }

  void loop(int w, uint64_t seen) {
    for (;;) {
      const std::function<void(int)>* job;
      {
        std::unique_lock<std::mutex> l(mu_);
        cv_.wait(l, [&] { return generation_ != seen; });
        seen = generation_;
        if (stopping_) return;
        job = job_;
      }
      (*job)(w);
      std::lock_guard<std::mutex> l(mu_);
      if (--pending_ == 0) done_cv_.notify_one();
    }
  }

  std::mutex call_mu_, mu_;
  std::condition_variable cv_, done_cv_;
  std::vector<std::thread> workers_;
  const std::function<void(int)>* job_ = nullptr;
  uint64_t generation_ = 0;
  int pending_ = 0;
  bool stopping_ = false;
};

Pool& pool() {
  static Pool p;
  return p;
}

int default_threads() {
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof(set), &set) == 0) return std::max(1, CPU_COUNT(&set));
  return std::max(1u, std::thread::hardware_concurrency());
}

// int16 columns per table entry: 4 per token, padded to whole 128-bit
// vectors for B > 1 (B = 1 uses one 64-bit half)
int64_t entry_lanes(int64_t B) { return B == 1 ? 4 : ((B + 1) / 2) * 8; }

struct Geometry {
  int64_t groups;        // K / 4
  int64_t lanes;         // int16 per entry
  int64_t window;        // groups per K window (multiple of kFlushGroups)
  size_t lut_bytes;
  size_t acc_bytes_per_thread;
};

Geometry geometry(int32_t T, int64_t K, int64_t B) {
  Geometry g;
  g.groups = K / 4;
  g.lanes = entry_lanes(B);
  const size_t group_bytes = 256 * static_cast<size_t>(g.lanes) * 2;
  int64_t w = static_cast<int64_t>(kWindowBytes / group_bytes);
  w = std::max<int64_t>(kFlushGroups, (w / kFlushGroups) * kFlushGroups);
  g.window = w;
  g.lut_bytes = static_cast<size_t>(g.groups) * group_bytes;
  g.acc_bytes_per_thread = static_cast<size_t>(kRowChunk) * 2 * T * g.lanes * 4;
  return g;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// contribution (four int16) of code c at a column with activation (qr, qi)
inline void code_contrib(int c, int16_t qr, int16_t qi, int16_t out[4]) {
  const int16_t s = (c & 2) ? -1 : 1;
  out[0] = out[1] = out[2] = out[3] = 0;
  if (c & 1) {
    out[2] = static_cast<int16_t>(s * qr);
    out[3] = static_cast<int16_t>(s * qi);
  } else {
    out[0] = static_cast<int16_t>(s * qr);
    out[1] = static_cast<int16_t>(s * qi);
  }
}

// table rows of groups [g0, g1) for every token
void build_lut(const int8_t* q, int64_t B, int64_t K, int64_t lanes, int16_t* lut, int64_t g0, int64_t g1) {
  for (int64_t g = g0; g < g1; ++g) {
    int16_t* row = lut + g * 256 * lanes;
    for (int64_t b = 0; b < B; ++b) {
      const int8_t* qb = q + (b * K + 4 * g) * 2;
      // half tables: lo over columns 0, 1 (index bits 0..3), hi over 2, 3
      int16_t lo[16][4], hi[16][4];
      for (int n = 0; n < 16; ++n) {
        int16_t a[4], c[4];
        code_contrib(n & 3, qb[0], qb[1], a);
        code_contrib(n >> 2, qb[2], qb[3], c);
        for (int v = 0; v < 4; ++v) lo[n][v] = static_cast<int16_t>(a[v] + c[v]);
        code_contrib(n & 3, qb[4], qb[5], a);
        code_contrib(n >> 2, qb[6], qb[7], c);
        for (int v = 0; v < 4; ++v) hi[n][v] = static_cast<int16_t>(a[v] + c[v]);
      }
      for (int idx = 0; idx < 256; ++idx) {
        int16_t* e = row + idx * lanes + 4 * b;
        for (int v = 0; v < 4; ++v) e[v] = static_cast<int16_t>(lo[idx & 15][v] + hi[idx >> 4][v]);
      }
    }
    if (lanes > 4 * B) {  // zero the padding lanes of odd B
      for (int idx = 0; idx < 256; ++idx)
        std::memset(row + idx * lanes + 4 * B, 0, (lanes - 4 * B) * sizeof(int16_t));
    }
  }
}

inline __m128i load_entry_b1(const int16_t* p) { return _mm_loadl_epi64(reinterpret_cast<const __m128i*>(p)); }
inline __m128i load_entry(const int16_t* p) { return _mm_loadu_si128(reinterpret_cast<const __m128i*>(p)); }

// add the sign-extended int16 lanes of v to the int32 array a[0 .. 8)
inline void widen_add(__m128i v, int32_t* a) {
  const __m128i lo = _mm_srai_epi32(_mm_unpacklo_epi16(v, v), 16);
  const __m128i hi = _mm_srai_epi32(_mm_unpackhi_epi16(v, v), 16);
  __m128i* p = reinterpret_cast<__m128i*>(a);
  _mm_storeu_si128(p, _mm_add_epi32(_mm_loadu_si128(p), lo));
  _mm_storeu_si128(p + 1, _mm_add_epi32(_mm_loadu_si128(p + 1), hi));
}

// One row, groups [g0, g0 + n) of one window, all P = 2T planes.  NV = 128-bit
// vectors per entry (0: B = 1, one 64-bit half).  acc: int32 [P][lanes].
template <int P, int NV>
void row_window(const uint8_t* const* plane_rows, const int16_t* lut, int64_t g0, int64_t n, int32_t* acc) {
  constexpr int kV = NV == 0 ? 1 : NV;
  constexpr int64_t lanes = NV == 0 ? 4 : 8 * NV;
  for (int64_t s = 0; s < n; s += kFlushGroups) {
    const int64_t e = std::min<int64_t>(n, s + kFlushGroups);
    __m128i a[P][kV];
    for (int p = 0; p < P; ++p)
      for (int v = 0; v < kV; ++v) a[p][v] = _mm_setzero_si128();
    for (int64_t g = g0 + s; g < g0 + e; ++g) {
      const int16_t* base = lut + g * 256 * lanes;
      for (int p = 0; p < P; ++p) {
        const int16_t* ent = base + static_cast<int64_t>(plane_rows[p][g]) * lanes;
        if constexpr (NV == 0) {
          a[p][0] = _mm_add_epi16(a[p][0], load_entry_b1(ent));
        } else {
          for (int v = 0; v < NV; ++v) a[p][v] = _mm_add_epi16(a[p][v], load_entry(ent + 8 * v));
        }
      }
    }
    for (int p = 0; p < P; ++p) {
      if constexpr (NV == 0) {
        // only the low four lanes are live
        const __m128i lo = _mm_srai_epi32(_mm_unpacklo_epi16(a[p][0], a[p][0]), 16);
        __m128i* q = reinterpret_cast<__m128i*>(acc + p * lanes);
        _mm_storeu_si128(q, _mm_add_epi32(_mm_loadu_si128(q), lo));
      } else {
        for (int v = 0; v < NV; ++v) widen_add(a[p][v], acc + p * lanes + 8 * v);
      }
    }
  }
}

using RowWindowFn = void (*)(const uint8_t* const*, const int16_t*, int64_t, int64_t, int32_t*);

template <int P>
RowWindowFn pick_nv(int64_t B) {
  if (B == 1) return row_window<P, 0>;
  switch ((B + 1) / 2) {
    case 1: return row_window<P, 1>;
    case 2: return row_window<P, 2>;
    case 3: return row_window<P, 3>;
    case 4: return row_window<P, 4>;
    case 5: return row_window<P, 5>;
    case 6: return row_window<P, 6>;
    case 7: return row_window<P, 7>;
    default: return row_window<P, 8>;
  }
}

RowWindowFn pick(int32_t T, int64_t B) {
  switch (T) {
    case 1: return pick_nv<2>(B);
    case 2: return pick_nv<4>(B);
    case 3: return pick_nv<6>(B);
    default: return pick_nv<8>(B);
  }
}

}  // namespace

extern "C" {

size_t fairy2i_cpu_lut_workspace_bytes(int32_t T, int64_t K, int64_t B, int32_t n_threads) {
  if (T < 1 || T > FAIRY2I_MAX_STAGES || K <= 0 || K % 4 != 0 || B < 1 || B > FAIRY2I_MAX_DECODE_BATCH) return 0;
  const int nt = n_threads > 0 ? std::min(n_threads, kMaxThreads) : std::min(default_threads(), kMaxThreads);
  const Geometry g = geometry(T, K, B);
  return align_up(g.lut_bytes, 64) + static_cast<size_t>(nt) * align_up(g.acc_bytes_per_thread, 64);
}

fairy2i_status fairy2i_cpu_lut_wl_matmul(const uint8_t* codes_U, const float* scales_U, const uint8_t* codes_W,
                                         const float* scales_W, int32_t T, int64_t N, int64_t K, const int8_t* q,
                                         const float* x_scale, int64_t B, float* y, int32_t* acc_out,
                                         void* workspace, size_t workspace_bytes, int32_t n_threads) {
  if (!codes_U || !codes_W || !q || !workspace || (!y && !acc_out)) return FAIRY2I_ERR_NULL;
  if (y && (!scales_U || !scales_W || !x_scale)) return FAIRY2I_ERR_NULL;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (N <= 0 || K <= 0 || K % 4 != 0 || B < 1 || B > FAIRY2I_MAX_DECODE_BATCH) return FAIRY2I_ERR_SHAPE;
  const int nt = n_threads > 0 ? std::min(n_threads, kMaxThreads) : std::min(default_threads(), kMaxThreads);
  if (workspace_bytes < fairy2i_cpu_lut_workspace_bytes(T, K, B, nt)) return FAIRY2I_ERR_WORKSPACE;

  const Geometry geo = geometry(T, K, B);
  const int P = 2 * T;
  int16_t* lut = static_cast<int16_t*>(workspace);
  char* acc_base = static_cast<char*>(workspace) + align_up(geo.lut_bytes, 64);
  const size_t acc_stride = align_up(geo.acc_bytes_per_thread, 64);
  const RowWindowFn fn = pick(T, B);
  const int64_t lanes = geo.lanes;
  const int64_t plane_bytes = N * (K / 4);
  const int64_t nchunks = (N + kRowChunk - 1) / kRowChunk;

  std::atomic<int64_t> next_group{0}, next_chunk{0};
  std::atomic<int> built{0};
  std::mutex bmu;
  std::condition_variable bcv;

  const std::function<void(int)> work = [&](int w) {
    // phase 1: the table, 16 groups at a time
    for (;;) {
      const int64_t g0 = next_group.fetch_add(16);
      if (g0 >= geo.groups) break;
      build_lut(q, B, K, lanes, lut, g0, std::min<int64_t>(geo.groups, g0 + 16));
    }
    {
      std::unique_lock<std::mutex> l(bmu);
      if (++built == nt) bcv.notify_all();
      else bcv.wait(l, [&] { return built.load() == nt; });
    }
    // phase 2: row chunks
    int32_t* acc = reinterpret_cast<int32_t*>(acc_base + w * acc_stride);
    for (;;) {
      const int64_t c = next_chunk.fetch_add(1);
      if (c >= nchunks) break;
      const int64_t r0 = c * kRowChunk;
      const int64_t nr = std::min<int64_t>(kRowChunk, N - r0);
      std::memset(acc, 0, static_cast<size_t>(nr) * P * lanes * sizeof(int32_t));
      for (int64_t g0 = 0; g0 < geo.groups; g0 += geo.window) {
        const int64_t n = std::min<int64_t>(geo.window, geo.groups - g0);
        for (int64_t r = 0; r < nr; ++r) {
          const uint8_t* rows[8];
          for (int m = 0; m < 2; ++m)
            for (int t = 0; t < T; ++t)
              rows[m * T + t] = (m == 0 ? codes_U : codes_W) + t * plane_bytes + (r0 + r) * (K / 4);
          fn(rows, lut, g0, n, acc + r * P * lanes);
        }
      }
      for (int64_t r = 0; r < nr; ++r) {
        const int64_t i = r0 + r;
        const int32_t* a = acc + r * P * lanes;
        if (acc_out) {
          // acc_out[M][t][p][b][i][c]
          for (int m = 0; m < 2; ++m)
            for (int t = 0; t < T; ++t)
              for (int64_t b = 0; b < B; ++b)
                for (int p = 0; p < 2; ++p)
                  for (int cc = 0; cc < 2; ++cc)
                    acc_out[(((static_cast<int64_t>(m) * T + t) * 2 + p) * B + b) * N * 2 + i * 2 + cc] =
                        a[(m * T + t) * lanes + 4 * b + 2 * p + cc];
        }
        if (y) {
          // Eq. (ifairy-dequant) applied to the axis sums, stages in order,
          // in double: U with q, W with conj(q); then the token factor
          for (int64_t b = 0; b < B; ++b) {
            double re = 0.0, im = 0.0;
            for (int t = 0; t < T; ++t) {
              const int32_t* u = a + t * lanes + 4 * b;
              const int32_t* v = a + (T + t) * lanes + 4 * b;
              const double su_re = scales_U[2 * t], su_im = scales_U[2 * t + 1];
              const double sw_re = scales_W[2 * t], sw_im = scales_W[2 * t + 1];
              const double tr = (su_re * u[0] - su_im * u[3]) + (sw_re * v[0] + sw_im * v[3]);
              const double ti = (su_re * u[1] + su_im * u[2]) + (-sw_re * v[1] + sw_im * v[2]);
              re += tr;
              im += ti;
            }
            const double f = x_scale[b];
            y[(b * N + i) * 2] = static_cast<float>(re * f);
            y[(b * N + i) * 2 + 1] = static_cast<float>(im * f);
          }
        }
      }
    }
  };
  pool().run(nt, work);
  return FAIRY2I_OK;
}

}  // extern "C"
