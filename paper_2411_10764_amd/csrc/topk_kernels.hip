// Selection of the k best accepted candidates (ML2Tuner Section 2: the
// explorer keeps the highest predicted performance among the configurations
// model V accepts, until (alpha+1)*N are held).
//
// Every included candidate i (mask set, score not NaN) gets a unique 64-bit
// key   (ord(score) << 32) | (0xFFFFFFFF - i)
// where ord maps float32 to uint32 monotonically (-0.0 first canonicalised to
// +0.0).  Larger keys are better: higher score, then lower index.  The k-th
// largest key is found by a most-significant-digit radix select over 12-bit
// digits.  A pool of at most kSmallN candidates is selected in one launch of
// one workgroup (topk_small: the included keys are gathered into LDS and the
// same digit passes run there).  Larger pools take three launches:
//   topk_init    clears the state and the digit histograms;
//   topk_select  one workgroup per CU at most, persistent over the pool: each
//                pass histograms (in LDS, then into a global histogram) the
//                digit below the decided prefix of the keys that match it;
//                after a grid-wide barrier every workgroup reads the
//                histogram and picks the same digit.  The passes stop once
//                the bin holding the k-th key is small (at most kInCap keys)
//                or holds exactly the keys still needed; one last pass over
//                the pool appends the keys above that bin (all selected) to
//                one list and the keys in it to another;
//   topk_finish  one workgroup: selects the needed keys of the bin in LDS
//                (the same digit passes over the bin's keys), sorts the k
//                selected keys (bitonic) and writes the outputs.
// The grid barrier waits a bounded time (every workgroup of the launch can
// be resident at once: the grid is at most one workgroup of 512 threads and
// 16 KiB of LDS per CU); a wait
// that runs out marks the selection failed (num_selected = -1) and every
// workgroup exits.
#include <math.h>

#include <mutex>
#include <vector>

#include "ml2_internal.h"

namespace ml2 {
namespace {

constexpr int kDigitBits = 12;
constexpr int kBins = 1 << kDigitBits;
constexpr int kMaxPasses = 6;    // 5 x 12 + 4 bits
constexpr int kSelThreads = 512;
constexpr int kSortThreads = 1024;
constexpr int kInCap = 8192;     // keys of the threshold bin finished in one workgroup
constexpr int kSmallN = 8192;    // pools selected in one launch of one workgroup
constexpr int kTile = 1024;      // candidates a wave reads per step (16 per lane)
constexpr size_t kStateBytes = 256;
constexpr size_t kHistBytes = 3 * kBins * sizeof(uint32_t);
constexpr double kBarrierSeconds = 2.0;

// How the final pass classifies keys.
constexpr int kTakeAll = 1;  // every included key is selected (#included <= k)
constexpr int kExact = 2;    // keys whose decided bits are >= prefix: exactly the k
constexpr int kInBin = 3;    // above prefix: selected; equal: the bin, need_in of them

struct TopkState {
  uint32_t arrive;   // grid-barrier arrivals in this call
  uint32_t failed;   // a barrier wait ran out
  uint32_t n_take;   // keys appended to the selected list
  uint32_t n_in;     // keys appended to the bin list
  int32_t k;
  int32_t total;     // included candidates
  int32_t mode;
  int32_t nbits;     // decided high bits
  int32_t need_in;   // keys of the bin to select
  int32_t pad;
  unsigned long long prefix;
};

__device__ __forceinline__ unsigned long long make_key(float s, int64_t i) {
  uint32_t b = __float_as_uint(s);
  if (b == 0x80000000u) b = 0u;
  const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((unsigned long long)ord << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)i);
}

__device__ __forceinline__ int digit_width(int nbits) { return min(kDigitBits, 64 - nbits); }

// f(included, key) for every candidate of this wave's share of the pool,
// called the same number of times by every lane of a wave (out-of-range
// candidates come as not included), so f may use wave ballots.  A wave reads
// kTile candidates per step: with 16-byte aligned scores (and a 4-byte
// aligned mask) four 16-byte score loads and four 4-byte mask loads per
// lane, each instruction covering 256 consecutive candidates, issued one
// step ahead of the step being processed; otherwise sixteen single loads
// per lane.
struct Tile {
  float4 s[4];
  uint32_t m[4];
};

__device__ __forceinline__ void load_tile(const uint8_t *valid, const float *scores, int64_t base,
                                          int lane, Tile &t) {
#pragma unroll
  for (int j = 0; j < 4; ++j)
    t.s[j] = reinterpret_cast<const float4 *>(scores + base)[j * 64 + lane];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    t.m[j] = valid ? reinterpret_cast<const uint32_t *>(valid + base)[j * 64 + lane] : 0x01010101u;
}

// f(inc[16], key[16]) for every group of 16 candidates of this wave's share
// of the pool (each lane's 16 of a tile of kTile), called the same number of
// times by every lane of a wave (out-of-range candidates come as not
// included), so f may use wave ballots.
template <typename F>
__device__ __forceinline__ void for_each_tile(const uint8_t *valid, const float *scores, int64_t n,
                                              int vec, F f) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int64_t full = vec ? n / kTile : 0;  // whole tiles read with vector loads
  int64_t t = wave;
  bool inc[16];
  unsigned long long key[16];
  for (; t < full; t += waves) {
    Tile cur;
    load_tile(valid, scores, t * kTile, lane, cur);
    const int64_t base = t * kTile;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i0 = base + 4 * (j * 64 + lane);
      const float c[4] = {cur.s[j].x, cur.s[j].y, cur.s[j].z, cur.s[j].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        inc[4 * j + q] = ((cur.m[j] >> (8 * q)) & 0xFFu) != 0 && !isnan(c[q]);
        key[4 * j + q] = make_key(c[q], i0 + q);
      }
    }
    f(inc, key);
  }
  // the rest (a partial tile, or every tile without vector loads)
  for (; t * kTile < n; t += waves) {
    const int64_t base = t * kTile;
#pragma unroll
    for (int j = 0; j < kTile / 64; ++j) {
      const int64_t i = base + j * 64 + lane;
      bool in = false;
      float sc = 0.0f;
      if (i < n) {
        sc = scores[i];
        in = (!valid || valid[i] != 0) && !isnan(sc);
      }
      inc[j] = in;
      key[j] = make_key(sc, i);
    }
    f(inc, key);
  }
}

// The digit holding the need-th largest key (1 <= need <= total) from a
// histogram h[nb] in LDS: bin, keys in higher bins, keys in the bin, and the
// histogram's total.  Every thread of the workgroup calls it; thread t
// covers bins from the top down.
struct Pick {
  int bin;
  uint32_t above, cnt, total;
};

__device__ __forceinline__ Pick block_pick(const uint32_t *h, int nb, uint32_t need, uint32_t *wave_sum,
                           Pick *out) {
  const int T = blockDim.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int per = nb / T > 0 ? nb / T : 1;
  const int hi = nb - t * per;  // bins [hi - per, hi)
  uint32_t sum = 0;
  for (int j = 1; j <= per; ++j)
    if (hi - j >= 0) sum += h[hi - j];
  uint32_t incl = sum;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t v = __shfl_up(incl, d);
    if (lane >= d) incl += v;
  }
  if (lane == 63) wave_sum[wave] = incl;
  __syncthreads();
  if (t == 0) {
    uint32_t acc = 0;
    for (int w = 0; w < (T >> 6); ++w) {
      const uint32_t v = wave_sum[w];
      wave_sum[w] = acc;
      acc += v;
    }
    wave_sum[T >> 6] = acc;
  }
  __syncthreads();
  incl += wave_sum[wave];
  const uint32_t excl = incl - sum;
  const uint32_t total = wave_sum[T >> 6];
  if (excl < need && need <= incl) {  // exactly one thread
    uint32_t c = excl;
    for (int j = 1; j <= per; ++j) {
      const int b = hi - j;
      if (c + h[b] >= need) {
        *out = Pick{b, c, h[b], total};
        break;
      }
      c += h[b];
    }
  }
  if (need > total && t == 0) *out = Pick{-1, 0, 0, total};
  __syncthreads();
  const Pick r = *out;
  __syncthreads();
  return r;
}

// Sort keys[0, size) descending in one workgroup of kSortThreads threads
// (bitonic network; size a power of two from 64 to 16 * kSortThreads; keys
// beyond the entries to sort are 0 and end up last).  Thread t holds the
// entries q * kSortThreads + t (t < size) in registers: a compare-exchange at
// distance 1024 or more stays in a thread, one below 64 goes through wave
// shuffles, and only the distances 64 .. 512 go through LDS (two barriers
// each); a size of 64 is sorted by the first wave alone, without barriers.
template <int Q>
__device__ __forceinline__ void block_sort_regs(unsigned long long *keys, int size) {
  const int t = threadIdx.x;
  const bool active = t < size;  // size < kSortThreads: whole waves idle
  unsigned long long r[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) r[q] = active ? keys[q * kSortThreads + t] : 0ull;
  for (int len = 2; len <= size; len <<= 1) {
    for (int stride = len >> 1; stride > 0; stride >>= 1) {
      if (stride >= kSortThreads) {
        const int qs = stride / kSortThreads;
#pragma unroll
        for (int c = 1; c < Q; c <<= 1) {  // c: the distance in registers, a constant
          if (qs == c) {
#pragma unroll
            for (int q = 0; q < Q; ++q) {
              if ((q & c) == 0) {
                const int j = q * kSortThreads + t;
                const bool desc = (j & len) == 0;
                const unsigned long long a = r[q], b = r[q | c];
                if (desc ? (a < b) : (a > b)) {
                  r[q] = b;
                  r[q | c] = a;
                }
              }
            }
          }
        }
      } else if (stride >= 64) {
        __syncthreads();
        if (active) {
#pragma unroll
          for (int q = 0; q < Q; ++q) keys[q * kSortThreads + t] = r[q];
        }
        __syncthreads();
        if (active) {
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            const int j = q * kSortThreads + t;
            const unsigned long long o = keys[j ^ stride];
            const bool lower = (j & stride) == 0;
            const bool desc = (j & len) == 0;
            const bool keep_max = lower == desc;
            r[q] = keep_max ? (r[q] > o ? r[q] : o) : (r[q] < o ? r[q] : o);
          }
        }
      } else if (active) {
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          const int j = q * kSortThreads + t;
          const uint32_t lo = __shfl_xor((uint32_t)r[q], stride);
          const uint32_t hi = __shfl_xor((uint32_t)(r[q] >> 32), stride);
          const unsigned long long o = ((unsigned long long)hi << 32) | lo;
          const bool lower = (j & stride) == 0;
          const bool desc = (j & len) == 0;
          const bool keep_max = lower == desc;
          r[q] = keep_max ? (r[q] > o ? r[q] : o) : (r[q] < o ? r[q] : o);
        }
      }
    }
  }
  __syncthreads();
  if (active) {
#pragma unroll
    for (int q = 0; q < Q; ++q) keys[q * kSortThreads + t] = r[q];
  }
  __syncthreads();
}

// keys[0, size) in LDS with size a power of two >= 64.
__device__ __forceinline__ void block_sort_desc(unsigned long long *keys, int size) {
  switch (size <= kSortThreads ? 1 : size / kSortThreads) {
    case 1: block_sort_regs<1>(keys, size); break;
    case 2: block_sort_regs<2>(keys, size); break;
    case 4: block_sort_regs<4>(keys, size); break;
    case 8: block_sort_regs<8>(keys, size); break;
    default: block_sort_regs<16>(keys, size); break;
  }
}

// Sort size of cnt keys: the next power of two, at least one wave.
__host__ __device__ constexpr int sort_size(int cnt) {
  int size = 64;
  while (size < cnt) size <<= 1;
  return size;
}

// Grid-wide barrier number `round` (1, 2, ...) of this call; false if the
// wait ran out (or another workgroup's did): the selection has failed.
__device__ __forceinline__ bool grid_sync(TopkState *st, uint32_t round, long long timeout_ticks, int *ok_s) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(&st->arrive, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t target = round * gridDim.x;
    const long long t0 = wall_clock64();
    int ok = 1;
    while (__hip_atomic_load(&st->arrive, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (__hip_atomic_load(&st->failed, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u ||
          wall_clock64() - t0 > timeout_ticks) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(4);
    }
    if (!ok) __hip_atomic_store(&st->failed, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *ok_s = ok;
  }
  // Only the waiting thread takes the acquire: what the workgroups read of
  // one another's writes (the digit histogram) is read with device-scope
  // atomic loads, and an acquire on every wave would invalidate the L2 once
  // per wave.
  __syncthreads();
  return *ok_s != 0;
}

// In one workgroup: of m keys (get(j), j < m) that share their top `nbits`
// bits (= prefix), the `need` largest (1 <= need <= m) are those whose top
// bits, on return, are >= prefix.  Digit passes over the keys with an LDS
// histogram, until the bin of the need-th key holds exactly the keys still
// needed (at the latest at 64 bits: keys are unique).
template <typename Get>
__device__ __forceinline__ void select_in_block(Get get, int m, uint32_t need, int &nbits,
                                unsigned long long &prefix, uint32_t *h, uint32_t *wave_sum,
                                Pick *pick_s) {
  const int T = blockDim.x;
  for (;;) {
    const int w = digit_width(nbits);
    const int shift = 64 - nbits - w;
    const unsigned long long dmask = (1ull << w) - 1ull;
    for (int b = threadIdx.x; b < kBins; b += T) h[b] = 0;
    __syncthreads();
    for (int j = threadIdx.x; j < m; j += T) {
      const unsigned long long key = get(j);
      if (nbits == 0 || (key >> (64 - nbits)) == prefix) atomicAdd(&h[(key >> shift) & dmask], 1u);
    }
    __syncthreads();
    const Pick p = block_pick(h, 1 << w, need, wave_sum, pick_s);
    need -= p.above;
    prefix = (nbits > 0 ? (prefix << w) : 0ull) | (unsigned long long)p.bin;
    nbits += w;
    if (p.cnt == need || nbits >= 64) return;
  }
}

__global__ void __launch_bounds__(256) topk_init(TopkState *st, uint32_t *hist, int32_t k) {
  for (int b = threadIdx.x; b < 3 * kBins; b += blockDim.x) hist[b] = 0;
  if (threadIdx.x == 0) {
    st->arrive = 0;
    st->failed = 0;
    st->n_take = 0;
    st->n_in = 0;
    st->k = k;
    st->total = 0;
    st->mode = 0;
    st->nbits = 0;
    st->need_in = 0;
    st->prefix = 0;
  }
}

__global__ void __launch_bounds__(kSelThreads) topk_select(
    const uint8_t *valid, const float *scores, int64_t n, int32_t k, int vec,
    long long timeout_ticks, TopkState *st, uint32_t *hist, unsigned long long *take,
    unsigned long long *inbin) {
  __shared__ uint32_t h[kBins];
  __shared__ uint32_t wave_sum[kSelThreads / 64 + 1];
  __shared__ Pick pick_s;
  __shared__ int ok_s;
  const int T = blockDim.x;
  const int lane = threadIdx.x & 63;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  unsigned long long prefix = 0ull;
  int nbits = 0;
  uint32_t need = (uint32_t)k;
  int mode = 0;
  for (int pass = 0; pass < kMaxPasses && mode == 0; ++pass) {
    const int w = digit_width(nbits);
    const int shift = 64 - nbits - w;
    const unsigned long long dmask = (1ull << w) - 1ull;
    for (int b = threadIdx.x; b < kBins; b += T) h[b] = 0;
    __syncthreads();
    for_each_tile(valid, scores, n, vec, [&](const bool *inc, const unsigned long long *key) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (inc[e] && (nbits == 0 || (key[e] >> (64 - nbits)) == prefix))
          atomicAdd(&h[(key[e] >> shift) & dmask], 1u);
    });
    __syncthreads();
    uint32_t *H = hist + (pass % 3) * kBins;
    for (int b = threadIdx.x; b < (1 << w); b += T)
      if (h[b]) atomicAdd(&H[b], h[b]);
    if (!grid_sync(st, (uint32_t)pass + 1, timeout_ticks, &ok_s)) return;
    for (int b = threadIdx.x; b < (1 << w); b += T)
      h[b] = __hip_atomic_load(&H[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the buffer two passes ahead was last read before this barrier
    if (blockIdx.x == 0)
      for (int b = threadIdx.x; b < kBins; b += T) hist[((pass + 2) % 3) * kBins + b] = 0;
    __syncthreads();
    const Pick p = block_pick(h, 1 << w, need, wave_sum, &pick_s);
    if (pass == 0) {  // every workgroup sums the same histogram
      if (blockIdx.x == 0 && threadIdx.x == 0) st->total = (int32_t)p.total;
      if (p.total <= need) {
        mode = kTakeAll;
        break;
      }
    }
    need -= p.above;
    prefix = (nbits > 0 ? (prefix << w) : 0ull) | (unsigned long long)p.bin;
    nbits += w;
    if (p.cnt == need)
      mode = kExact;
    else if (p.cnt <= (uint32_t)kInCap)
      mode = kInBin;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->mode = mode;
    st->nbits = nbits;
    st->prefix = prefix;
    st->need_in = (int32_t)need;
  }
  // the final pass: selected keys and the bin's keys, appended per wave;
  // a group of 16 candidates of which no lane selects any costs one ballot
  for_each_tile(valid, scores, n, vec, [&](const bool *inc, const unsigned long long *key) {
    int cls[16];  // 1 selected, 2 in the bin
    bool any = false;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      cls[e] = 0;
      if (inc[e]) {
        if (mode == kTakeAll) {
          cls[e] = 1;
        } else {
          const unsigned long long top = key[e] >> (64 - nbits);
          cls[e] = top > prefix ? 1 : top == prefix ? (mode == kExact ? 1 : 2) : 0;
        }
      }
      any = any || cls[e] != 0;
    }
    if (__ballot(any) == 0) return;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint64_t b1 = __ballot(cls[e] == 1);
      if (b1) {
        uint32_t p0 = 0;
        if (lane == 0) p0 = atomicAdd(&st->n_take, (uint32_t)__popcll(b1));
        p0 = __shfl(p0, 0);
        if (cls[e] == 1) {
          const uint32_t pos = p0 + (uint32_t)__popcll(b1 & below);
          if (pos < (uint32_t)k) take[pos] = key[e];
        }
      }
      const uint64_t b2 = __ballot(cls[e] == 2);
      if (b2) {
        uint32_t p0 = 0;
        if (lane == 0) p0 = atomicAdd(&st->n_in, (uint32_t)__popcll(b2));
        p0 = __shfl(p0, 0);
        if (cls[e] == 2) {
          const uint32_t pos = p0 + (uint32_t)__popcll(b2 & below);
          if (pos < (uint32_t)kInCap) inbin[pos] = key[e];
        }
      }
    }
  });
}

// One workgroup: the keys of the bin still needed (digit passes in LDS over
// the bin's list), then the k selected keys sorted descending, then the
// outputs.  keys: the selected keys (next power of two of k entries).
__global__ void __launch_bounds__(kSortThreads) topk_finish(const float *scores, int64_t n,
                                                            const TopkState *st,
                                                            const unsigned long long *take,
                                                            const unsigned long long *inbin,
                                                            int32_t *idx, float *out,
                                                            int32_t *num) {
  extern __shared__ unsigned long long keys[];
  __shared__ uint32_t h[kBins];
  __shared__ uint32_t wave_sum[kSortThreads / 64 + 1];
  __shared__ Pick pick_s;
  __shared__ uint32_t fill_s;
  const int T = blockDim.x;
  const int k = st->k;
  if (st->failed) {
    for (int j = threadIdx.x; j < k; j += T) {
      idx[j] = -1;
      out[j] = -INFINITY;
    }
    if (threadIdx.x == 0) *num = -1;
    return;
  }
  const int mode = st->mode;
  const int cnt = (mode == 0) ? 0 : min(k, st->total);
  const int nt = (mode == 0) ? 0 : (int)min(st->n_take, (uint32_t)k);
  const int size = sort_size(cnt);
  for (int j = threadIdx.x; j < size; j += T) keys[j] = (j < nt) ? take[j] : 0ull;
  if (mode == kInBin) {
    // the need_in largest of the m keys of the bin, which share the top nbits
    const int m = (int)min(st->n_in, (uint32_t)kInCap);
    int nbits = st->nbits;
    unsigned long long prefix = st->prefix;
    select_in_block([&](int j) { return inbin[j]; }, m, (uint32_t)st->need_in, nbits, prefix, h,
                    wave_sum, &pick_s);
    if (threadIdx.x == 0) fill_s = 0;
    __syncthreads();
    for (int j = threadIdx.x; j < m; j += T) {
      const unsigned long long key = inbin[j];
      if ((key >> (64 - nbits)) >= prefix) {
        const uint32_t pos = atomicAdd(&fill_s, 1u);
        if (nt + (int)pos < size) keys[nt + pos] = key;
      }
    }
  }
  __syncthreads();
  block_sort_desc(keys, size);
  for (int j = threadIdx.x; j < k; j += T) {
    const int64_t i = (int64_t)(0xFFFFFFFFu - (uint32_t)(keys[j] & 0xFFFFFFFFull));
    if (j < cnt && keys[j] != 0ull && i < n) {  // (always, for a selection that completed)
      idx[j] = (int32_t)i;
      out[j] = scores[i];
    } else {
      idx[j] = -1;
      out[j] = -INFINITY;
    }
  }
  if (threadIdx.x == 0) *num = cnt;
}

// Pools of at most kSmallN candidates, in one launch of one workgroup: the
// included keys are gathered into LDS, the k largest selected there (digit
// passes) and sorted.  LDS: the sort area (sort_size(min(k, n)) keys), then
// the gathered keys (n).
__global__ void __launch_bounds__(kSortThreads) topk_small(const uint8_t *valid,
                                                           const float *scores, int64_t n,
                                                           int32_t k, int32_t *idx, float *out,
                                                           int32_t *num) {
  extern __shared__ unsigned long long lds_keys[];
  __shared__ uint32_t h[kBins];
  __shared__ uint32_t wave_sum[kSortThreads / 64 + 1];
  __shared__ Pick pick_s;
  __shared__ uint32_t cnt_s, fill_s;
  const int T = blockDim.x;
  const int lane = threadIdx.x & 63;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int nn = (int)n;
  const int size = sort_size(min(k, nn));
  unsigned long long *B = lds_keys;
  unsigned long long *A = lds_keys + size;
  if (threadIdx.x == 0) {
    cnt_s = 0;
    fill_s = 0;
  }
  for (int j = threadIdx.x; j < size; j += T) B[j] = 0ull;
  __syncthreads();
  for (int base = 0; base < nn; base += T) {  // uniform trip count: ballots below
    const int i = base + threadIdx.x;
    bool inc = false;
    float sc = 0.0f;
    if (i < nn) {
      sc = scores[i];
      inc = (!valid || valid[i] != 0) && !isnan(sc);
    }
    const uint64_t bal = __ballot(inc);
    if (bal) {
      uint32_t p0 = 0;
      if (lane == 0) p0 = atomicAdd(&cnt_s, (uint32_t)__popcll(bal));
      p0 = __shfl(p0, 0);
      if (inc) A[p0 + __popcll(bal & below)] = make_key(sc, i);
    }
  }
  __syncthreads();
  const int m = (int)cnt_s;
  const int cnt = min(k, m);
  if (m <= k) {
    for (int j = threadIdx.x; j < m; j += T) B[j] = A[j];
  } else if (cnt > 0) {
    int nbits = 0;
    unsigned long long prefix = 0ull;
    select_in_block([&](int j) { return A[j]; }, m, (uint32_t)k, nbits, prefix, h, wave_sum,
                    &pick_s);
    for (int j = threadIdx.x; j < m; j += T) {
      const unsigned long long key = A[j];
      if ((key >> (64 - nbits)) >= prefix) {
        const uint32_t pos = atomicAdd(&fill_s, 1u);
        if ((int)pos < size) B[pos] = key;
      }
    }
  }
  __syncthreads();
  block_sort_desc(B, size);
  for (int j = threadIdx.x; j < k; j += T) {
    const int64_t i = (int64_t)(0xFFFFFFFFu - (uint32_t)(B[j] & 0xFFFFFFFFull));
    if (j < cnt && B[j] != 0ull && i < n) {
      idx[j] = (int32_t)i;
      out[j] = scores[i];
    } else {
      idx[j] = -1;
      out[j] = -INFINITY;
    }
  }
  if (threadIdx.x == 0) *num = cnt;
}

// Float32 of an order-preserving key's high word (inverse of make_key's map;
// a zero comes back as +0.0).
__device__ __forceinline__ float key_score(unsigned long long key) {
  const uint32_t ord = (uint32_t)(key >> 32);
  const uint32_t b = (ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord;
  return __uint_as_float(b);
}

// Key of a listed row for the second-level selection: the high word orders
// by score (-0.0 and +0.0 equal), the low word by pool row ascending
// (0x7FFFFFFF - row, row < 2^31, in bits 31..1) and keeps, in bit 0, the
// sign of a zero score, so that the chosen entry's score comes back bit for
// bit.  Two entries of one row carry the same score (the same row walked by
// the same model), so bit 0 never reorders distinct scores.
__device__ __forceinline__ unsigned long long row_key(float s, int32_t row) {
  const uint32_t neg_zero = (__float_as_uint(s) == 0x80000000u) ? 1u : 0u;
  const uint32_t lo = ((0x7FFFFFFFu - (uint32_t)row) << 1) | neg_zero;
  return (make_key(s, 0) & 0xFFFFFFFF00000000ull) | (unsigned long long)lo;
}
__device__ __forceinline__ int32_t row_key_row(unsigned long long key) {
  return (int32_t)(0x7FFFFFFFu - ((uint32_t)key >> 1));
}
__device__ __forceinline__ float row_key_score(unsigned long long key) {
  return (key & 1ull) ? -0.0f : key_score(key);
}

// Second-level selection (model A): one workgroup sorts the keys of the m
// listed rows (row_key) and writes the best `keep`.  Rows outside [0, n)
// and NaN scores are left out (key 0, below every included key: a zero high
// word is the ord of a negative NaN).
__global__ void __launch_bounds__(kSortThreads) rerank_select(const int32_t *rows,
                                                              const float *scores, int32_t m,
                                                              int64_t n, int32_t keep,
                                                              int32_t *idx, float *out,
                                                              int32_t *num) {
  extern __shared__ unsigned long long keys[];
  __shared__ int included_s;
  if (threadIdx.x == 0) included_s = 0;
  const int size = sort_size(m);
  __syncthreads();
  int mine = 0;
  for (int j = threadIdx.x; j < size; j += blockDim.x) {
    unsigned long long key = 0ull;
    if (j < m) {
      const int32_t r = rows[j];
      const float sc = scores[j];
      if (r >= 0 && r < n && !isnan(sc)) {
        key = row_key(sc, r);
        ++mine;
      }
    }
    keys[j] = key;
  }
  if (mine) atomicAdd(&included_s, mine);
  __syncthreads();
  block_sort_desc(keys, size);
  const int cnt = min(included_s, keep);
  for (int j = threadIdx.x; j < keep; j += blockDim.x) {
    if (j < cnt) {
      idx[j] = row_key_row(keys[j]);
      out[j] = row_key_score(keys[j]);
    } else {
      idx[j] = -1;
      out[j] = -INFINITY;
    }
  }
  if (threadIdx.x == 0) *num = cnt;
}

// Rows already proposed leave the pool: mask[rows[j]] = 0 for the listed rows
// inside [0, n) (the -1 padding of short rounds is skipped).
__global__ void __launch_bounds__(256) exclude_rows(uint8_t *mask, int64_t n,
                                                    const int32_t *rows, int32_t m) {
  const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  const int32_t r = rows[j];
  if (r >= 0 && r < n) mask[r] = 0;
}

// A chunk of pool rows row0 .. row0+m-1 (streamed explorer): rows proposed in
// earlier rounds leave the chunk's mask, mask[r - row0] = 0 for every listed
// row r inside the chunk (the -1 padding of short rounds never is).
__global__ void __launch_bounds__(256) exclude_range(uint8_t *mask, int64_t row0, int64_t m,
                                                     const int32_t *rows, int32_t count) {
  const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= count) return;
  const int64_t r = rows[j];
  if (r >= row0 && r < row0 + m) mask[r - row0] = 0;
}

// An empty held set: no rows, every slot -1 / -inf.
__global__ void __launch_bounds__(256) held_reset(int32_t *held_id, float *held_p,
                                                  float *held_a, int32_t *held_n, int32_t k) {
  for (int32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < k; j += gridDim.x * blockDim.x) {
    held_id[j] = -1;
    held_p[j] = -INFINITY;
    held_a[j] = -INFINITY;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *held_n = 0;
}

// The held set of the streamed explorer after one more chunk: the k best of
// the rows held so far (h_*, *h_n of them) and the chunk's selection (c_*,
// *c_n of them, chunk-local indices; pool row = row0 + index) by (P score
// desc, pool row asc), a row present in both counted once.  Each entry
// carries its P score and its second-level score (model A's, or P's again
// when c_a is NULL), copied bit for bit.  One workgroup: keys
// (ord(P) << 32) | (0xFFFFFFFF - row) and their source positions are sorted
// together in LDS (bitonic, descending); equal keys are the same row with the
// same score, so every key after an equal one is dropped.
__global__ void __launch_bounds__(kSortThreads) merge_held(
    const int32_t *h_id, const float *h_p, const float *h_a, const int32_t *h_n,
    const int32_t *c_idx, const float *c_p, const float *c_a, const int32_t *c_n, int64_t row0,
    int32_t k, int32_t *o_id, float *o_p, float *o_a, int32_t *o_n) {
  extern __shared__ unsigned long long keys[];
  __shared__ int warp_sum[kSortThreads / 64 + 1];
  int size = 1;
  while (size < 2 * k) size <<= 1;
  int32_t *pos = reinterpret_cast<int32_t *>(keys + size);
  const int hn = min(*h_n, k), cn = min(*c_n, k);
  for (int j = threadIdx.x; j < size; j += blockDim.x) {
    unsigned long long key = 0ull;
    if (j < hn) {
      key = make_key(h_p[j], h_id[j]);
    } else if (j >= k && j - k < cn) {
      key = make_key(c_p[j - k], row0 + c_idx[j - k]);
    }
    keys[j] = key;
    pos[j] = j;
  }
  __syncthreads();
  for (int len = 2; len <= size; len <<= 1) {
    for (int stride = len >> 1; stride > 0; stride >>= 1) {
      for (int j = threadIdx.x; j < size; j += blockDim.x) {
        const int p = j ^ stride;
        if (p > j) {
          const unsigned long long a = keys[j], b = keys[p];
          const bool desc = (j & len) == 0;
          if (desc ? (a < b) : (a > b)) {
            keys[j] = b;
            keys[p] = a;
            const int32_t t = pos[j];
            pos[j] = pos[p];
            pos[p] = t;
          }
        }
      }
      __syncthreads();
    }
  }
  // Rank of each first occurrence: each thread owns a run of consecutive
  // sorted entries; the runs' counts are scanned across the workgroup.
  const int per = size / blockDim.x > 0 ? size / blockDim.x : 1;
  const int lo = threadIdx.x * per;
  const bool owner = lo < size;
  int mine = 0;
  if (owner)
    for (int j = lo; j < lo + per; ++j)
      mine += (keys[j] != 0ull && (j == 0 || keys[j] != keys[j - 1])) ? 1 : 0;
  // inclusive scan of `mine` over the threads: waves, then wave totals
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = mine;
  for (int d = 1; d < 64; d <<= 1) {
    const int v = __shfl_up(incl, d);
    if (lane >= d) incl += v;
  }
  if (lane == 63) warp_sum[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      const int t = warp_sum[w];
      warp_sum[w] = acc;
      acc += t;
    }
    warp_sum[blockDim.x >> 6] = acc;
  }
  __syncthreads();
  const int unique = warp_sum[blockDim.x >> 6];
  if (owner) {
    int r = warp_sum[wave] + incl - mine;  // rank of this run's first occurrence
    for (int j = lo; j < lo + per; ++j) {
      if (keys[j] == 0ull || (j > 0 && keys[j] == keys[j - 1])) continue;
      if (r < k) {
        const int src = pos[j];
        if (src < k) {
          o_id[r] = h_id[src];
          o_p[r] = h_p[src];
          o_a[r] = h_a[src];
        } else {
          const int c = src - k;
          o_id[r] = (int32_t)(row0 + c_idx[c]);
          o_p[r] = c_p[c];
          o_a[r] = c_a ? c_a[c] : c_p[c];
        }
      }
      ++r;
    }
  }
  const int held = min(unique, k);
  for (int r = held + threadIdx.x; r < k; r += blockDim.x) {
    o_id[r] = -1;
    o_p[r] = -INFINITY;
    o_a[r] = -INFINITY;
  }
  if (threadIdx.x == 0) *o_n = held;
}

}  // namespace

// Workspace: state, three digit histograms, the selected list (k keys) and
// the threshold bin's list (kInCap keys).  Independent of n.
size_t topk_workspace_bytes(int64_t n, int32_t k) {
  (void)n;
  const size_t take = (size_t)(k > 0 ? k : 1) * sizeof(unsigned long long);
  const size_t inbin = (size_t)kInCap * sizeof(unsigned long long);
  return (kStateBytes + kHistBytes + take + inbin + 255) & ~(size_t)255;
}

// The selection's workspace for callers that cannot allocate
// (ml2_filter_topk_noalloc): one file-scope array per device, sized for the
// largest k, shared by every such call on that device.  Host code never
// passes `scratch` itself to a kernel (on the host it only names the
// symbol); it uses the device address hipGetSymbolAddress returns, taken
// once per device with that device current.
constexpr size_t kStaticScratchBytes =
    (kStateBytes + kHistBytes + (size_t)(ML2_MAX_TOPK + kInCap) * sizeof(unsigned long long) +
     255) &
    ~(size_t)255;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch(int device, void **ptr) {
  static std::mutex mu;
  static std::vector<void *> addr;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)addr.size() <= device) addr.resize((size_t)device + 1, nullptr);
  if (!addr[(size_t)device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255u)) return hipErrorInvalidSymbol;
    addr[(size_t)device] = p;
  }
  *ptr = addr[(size_t)device];
  return hipSuccess;
}

namespace {

// Wall-clock ticks of the grid barrier's longest wait, per device.
hipError_t barrier_ticks(long long *ticks) {
  static std::mutex mu;
  static std::vector<long long> cache;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) cache.resize((size_t)dev + 1, 0);
  if (cache[(size_t)dev] == 0) {
    int khz = 0;
    e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return e;
    if (khz <= 0) khz = 100000;  // the 100 MHz constant clock
    cache[(size_t)dev] = (long long)(kBarrierSeconds * 1000.0 * khz);
  }
  *ticks = cache[(size_t)dev];
  return hipSuccess;
}


}  // namespace

hipError_t launch_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                       int32_t *idx, float *score, int32_t *num, void *ws, int cu_count,
                       hipStream_t s) {
  char *w = static_cast<char *>(ws);
  TopkState *st = reinterpret_cast<TopkState *>(w);
  uint32_t *hist = reinterpret_cast<uint32_t *>(w + kStateBytes);
  unsigned long long *take =
      reinterpret_cast<unsigned long long *>(w + kStateBytes + kHistBytes);
  unsigned long long *inbin = take + (k > 0 ? k : 1);
  if (n <= kSmallN) {
    const size_t lds =
        ((size_t)sort_size(min((int64_t)k, n)) + (size_t)(n > 0 ? n : 1)) * sizeof(unsigned long long);
    const size_t most = ((size_t)sort_size(kSmallN) + kSmallN) * sizeof(unsigned long long);
    hipError_t e = ensure_dynamic_lds(reinterpret_cast<const void *>(&topk_small), most);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(topk_small, dim3(1), dim3(kSortThreads), lds, s, valid, scores, n, k, idx,
                       score, num);
    return hipGetLastError();
  }
  long long ticks = 0;
  hipError_t e = barrier_ticks(&ticks);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_init, dim3(1), dim3(256), 0, s, st, hist, k);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n > 0 && k > 0) {
    const int vec = ((reinterpret_cast<uintptr_t>(scores) & 15u) == 0 &&
                     (reinterpret_cast<uintptr_t>(valid) & 3u) == 0)
                        ? 1
                        : 0;
    const int64_t per_wg = (int64_t)kTile * (kSelThreads / 64);
    int64_t grid = (n + per_wg - 1) / per_wg;
    if (grid > cu_count) grid = cu_count;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(topk_select, dim3((unsigned)grid), dim3(kSelThreads), 0, s, valid, scores,
                       n, k, vec, ticks, st, hist, take, inbin);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t lds = (size_t)sort_size(k) * sizeof(unsigned long long);
  e = ensure_dynamic_lds(reinterpret_cast<const void *>(&topk_finish), lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_finish, dim3(1), dim3(kSortThreads), lds, s, scores, n, st, take,
                     inbin, idx, score, num);
  return hipGetLastError();
}

hipError_t launch_rerank_select(const int32_t *rows, const float *scores, int32_t m, int64_t n,
                                int32_t keep, int32_t *idx, float *score, int32_t *num,
                                hipStream_t s) {
  const size_t lds = (size_t)sort_size(m) * sizeof(unsigned long long);
  hipError_t e = ensure_dynamic_lds(reinterpret_cast<const void *>(&rerank_select), lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(rerank_select, dim3(1), dim3(kSortThreads), lds, s, rows, scores, m, n, keep,
                     idx, score, num);
  return hipGetLastError();
}

hipError_t launch_exclude(uint8_t *mask, int64_t n, const int32_t *rows, int32_t m,
                          hipStream_t s) {
  if (m <= 0) return hipSuccess;
  hipLaunchKernelGGL(exclude_rows, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, s, mask, n,
                     rows, m);
  return hipGetLastError();
}

hipError_t launch_exclude_range(uint8_t *mask, int64_t row0, int64_t m, const int32_t *rows,
                                int32_t count, hipStream_t s) {
  if (count <= 0 || m <= 0) return hipSuccess;
  hipLaunchKernelGGL(exclude_range, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, mask,
                     row0, m, rows, count);
  return hipGetLastError();
}

hipError_t launch_held_reset(int32_t *held_id, float *held_p, float *held_a, int32_t *held_n,
                             int32_t k, hipStream_t s) {
  hipLaunchKernelGGL(held_reset, dim3((unsigned)((k + 255) / 256)), dim3(256), 0, s, held_id,
                     held_p, held_a, held_n, k);
  return hipGetLastError();
}

size_t merge_held_lds(int32_t k) {
  int size = 1;
  while (size < 2 * k) size <<= 1;
  return (size_t)size * (sizeof(unsigned long long) + sizeof(int32_t));
}

hipError_t launch_merge_held(const int32_t *h_id, const float *h_p, const float *h_a,
                             const int32_t *h_n, const int32_t *c_idx, const float *c_p,
                             const float *c_a, const int32_t *c_n, int64_t row0, int32_t k,
                             int32_t *o_id, float *o_p, float *o_a, int32_t *o_n, hipStream_t s) {
  const size_t lds = merge_held_lds(k);
  hipError_t e = ensure_dynamic_lds(reinterpret_cast<const void *>(&merge_held), lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_held, dim3(1), dim3(kSortThreads), lds, s, h_id, h_p, h_a, h_n, c_idx,
                     c_p, c_a, c_n, row0, k, o_id, o_p, o_a, o_n);
  return hipGetLastError();
}

}  // namespace ml2
