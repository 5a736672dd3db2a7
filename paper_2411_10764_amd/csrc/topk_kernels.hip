// Selection of the k best accepted candidates (ML2Tuner Section 2: the
// explorer keeps the highest predicted performance among the configurations
// model V accepts, until (alpha+1)*N are held).
//
// Every included candidate i (mask set, score not NaN) gets a unique 64-bit
// key   (ord(score) << 32) | (0xFFFFFFFF - i)
// where ord maps float32 to uint32 monotonically (-0.0 first canonicalised to
// +0.0).  Larger keys are better: higher score, then lower index.  The k-th
// largest key is found by a most-significant-digit radix select (12-bit
// digits; each pass histograms the candidates that still match the chosen
// prefix and fixes one more digit), stopping as soon as the threshold bucket
// holds exactly the number still needed.  A final pass gathers the keys above
// the threshold (exactly min(k, #included) of them) and one workgroup sorts
// them (bitonic, in LDS).  Every pass is launched unconditionally and exits at
// once when the selection is already complete, so the host never waits.
#include <math.h>

#include <mutex>
#include <vector>

#include "ml2_internal.h"

namespace ml2 {
namespace {

constexpr int kDigitBits = 12;
constexpr int kBins = 1 << kDigitBits;
constexpr int kPasses = 6;  // 5 x 12 + 4 bits
constexpr int kSortThreads = 1024;
constexpr size_t kStateBytes = 256;
constexpr size_t kHistBytes = kBins * sizeof(uint32_t);

struct TopkState {
  unsigned long long prefix;  // decided high bits of the threshold key
  int nbits;                  // how many high bits are decided
  int need;                   // keys still to take among those matching prefix
  int done;                   // selection criterion complete
  int total;                  // included candidates
  int count;                  // gathered keys
  int k;
};

__device__ __forceinline__ bool included(const uint8_t *valid, const float *scores, int64_t i,
                                         float *s) {
  if (valid && valid[i] == 0) return false;
  *s = scores[i];
  return !isnan(*s);
}

__device__ __forceinline__ unsigned long long make_key(float s, int64_t i) {
  uint32_t b = __float_as_uint(s);
  if (b == 0x80000000u) b = 0u;
  const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((unsigned long long)ord << 32) | (unsigned long long)(0xFFFFFFFFu - (uint32_t)i);
}

__global__ void topk_init(TopkState *st, uint32_t *hist, int32_t k, int64_t n) {
  for (int b = threadIdx.x; b < kBins; b += blockDim.x) hist[b] = 0;
  if (threadIdx.x == 0) {
    st->prefix = 0;
    st->nbits = 0;
    st->need = k;
    st->done = (k == 0 || n == 0) ? 1 : 0;
    st->total = 0;
    st->count = 0;
    st->k = k;
  }
}

// Histogram of the next digit over candidates matching the decided prefix.
__global__ void __launch_bounds__(256) topk_hist(const uint8_t *valid, const float *scores,
                                                 int64_t n, const TopkState *st, uint32_t *hist) {
  __shared__ uint32_t h[kBins];
  if (st->done) return;
  const int nbits = st->nbits;
  const unsigned long long prefix = st->prefix;
  const int w = min(kDigitBits, 64 - nbits);
  const int shift = 64 - nbits - w;
  const unsigned long long dmask = (1ull << w) - 1ull;
  for (int b = threadIdx.x; b < kBins; b += blockDim.x) h[b] = 0;
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    float s;
    if (!included(valid, scores, i, &s)) continue;
    const unsigned long long key = make_key(s, i);
    if (nbits > 0 && (key >> (64 - nbits)) != prefix) continue;
    atomicAdd(&h[(key >> shift) & dmask], 1u);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < kBins; b += blockDim.x)
    if (h[b]) atomicAdd(&hist[b], h[b]);
}

// One workgroup: pick the digit holding the need-th largest key, update the
// state, clear the histogram for the next pass.
__global__ void __launch_bounds__(256) topk_pick(TopkState *st, uint32_t *hist, int pass) {
  __shared__ uint32_t part[256];
  __shared__ int total_s;
  if (st->done) return;
  const int nbits = st->nbits;
  const int w = min(kDigitBits, 64 - nbits);
  const int nb = 1 << w;
  const int per = (nb + 255) / 256;  // bins per thread, from the top down
  const int t = threadIdx.x;
  // thread t owns bins [nb - (t+1)*per, nb - t*per) (the highest bins first)
  uint32_t sum = 0;
  for (int j = 0; j < per; ++j) {
    const int b = nb - 1 - (t * per + j);
    if (b >= 0) sum += hist[b];
  }
  part[t] = sum;
  __syncthreads();
  if (t == 0) {
    uint32_t tot = 0;
    for (int j = 0; j < 256; ++j) tot += part[j];
    total_s = (int)tot;
  }
  __syncthreads();
  if (t == 0) {
    int need = st->need;
    if (pass == 0) {
      st->total = total_s;
      if (total_s <= need) {  // everything included is selected
        st->need = total_s;
        st->done = 1;
        need = -1;
      }
    }
    if (need > 0) {
      uint32_t cum = 0;
      int owner = 0;
      for (; owner < 256; ++owner) {
        if (cum + part[owner] >= (uint32_t)need) break;
        cum += part[owner];
      }
      int chosen = -1;
      uint32_t inb = 0;
      for (int j = 0; j < per; ++j) {
        const int b = nb - 1 - (owner * per + j);
        if (b < 0) break;
        if (cum + hist[b] >= (uint32_t)need) {
          chosen = b;
          inb = hist[b];
          break;
        }
        cum += hist[b];
      }
      need -= (int)cum;
      st->prefix = (nbits > 0 ? (st->prefix << w) : 0ull) | (unsigned long long)chosen;
      st->nbits = nbits + w;
      st->need = need;
      if ((uint32_t)need == inb || nbits + w >= 64) st->done = 1;
    }
  }
  __syncthreads();
  for (int b = t; b < kBins; b += blockDim.x) hist[b] = 0;
}

// Gather every included key whose decided high bits are >= the prefix.
__global__ void __launch_bounds__(256) topk_gather(const uint8_t *valid, const float *scores,
                                                   int64_t n, TopkState *st,
                                                   unsigned long long *cand) {
  const int k = st->k;
  if (k == 0) return;
  const int nbits = st->nbits;
  const unsigned long long prefix = st->prefix;
  const int lane = threadIdx.x & 63;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t start = (int64_t)blockIdx.x * blockDim.x;
  for (int64_t base = start; base < n; base += stride) {  // uniform trip count per wave
    const int64_t i = base + threadIdx.x;
    bool take = false;
    unsigned long long key = 0;
    float s;
    if (i < n && included(valid, scores, i, &s)) {
      key = make_key(s, i);
      take = (nbits == 0) || ((key >> (64 - nbits)) >= prefix);
    }
    const uint64_t bal = __ballot(take);
    if (bal == 0) continue;
    int pos0 = 0;
    if (lane == 0) pos0 = atomicAdd(&st->count, __popcll(bal));
    pos0 = __shfl(pos0, 0);
    if (take) {
      const int pos = pos0 + __popcll(bal & below);
      if (pos < k) cand[pos] = key;
    }
  }
}

// One workgroup: sort the gathered keys descending and write the outputs.
__global__ void __launch_bounds__(kSortThreads) topk_sort(const float *scores, TopkState *st,
                                                          const unsigned long long *cand,
                                                          int32_t *idx, float *out,
                                                          int32_t *num) {
  extern __shared__ unsigned long long keys[];
  const int k = st->k;
  const int cnt = min(st->count, k);
  int size = 1;
  while (size < cnt) size <<= 1;
  for (int j = threadIdx.x; j < size; j += blockDim.x) keys[j] = (j < cnt) ? cand[j] : 0ull;
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
          }
        }
      }
      __syncthreads();
    }
  }
  for (int j = threadIdx.x; j < k; j += blockDim.x) {
    if (j < cnt) {
      const int32_t i = (int32_t)(0xFFFFFFFFu - (uint32_t)(keys[j] & 0xFFFFFFFFull));
      idx[j] = i;
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
  int size = 1;
  while (size < m) size <<= 1;
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
          }
        }
      }
      __syncthreads();
    }
  }
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

size_t topk_workspace_bytes(int64_t n, int32_t k) {
  (void)n;
  const size_t cand = (size_t)(k > 0 ? k : 1) * sizeof(unsigned long long);
  return (kStateBytes + kHistBytes + cand + 255) & ~(size_t)255;
}

// The selection's workspace for callers that cannot allocate
// (ml2_filter_topk_noalloc): one file-scope array per device, sized for the
// largest k, shared by every such call on that device.  Host code never
// passes `scratch` itself to a kernel (on the host it only names the
// symbol); it uses the device address hipGetSymbolAddress returns, taken
// once per device with that device current.
constexpr size_t kStaticScratchBytes =
    (kStateBytes + kHistBytes + (size_t)ML2_MAX_TOPK * sizeof(unsigned long long) + 255) &
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

hipError_t launch_topk(const uint8_t *valid, const float *scores, int64_t n, int32_t k,
                       int32_t *idx, float *score, int32_t *num, void *ws, int cu_count,
                       hipStream_t s) {
  char *w = static_cast<char *>(ws);
  TopkState *st = reinterpret_cast<TopkState *>(w);
  uint32_t *hist = reinterpret_cast<uint32_t *>(w + kStateBytes);
  unsigned long long *cand = reinterpret_cast<unsigned long long *>(w + kStateBytes + kHistBytes);
  hipLaunchKernelGGL(topk_init, dim3(1), dim3(256), 0, s, st, hist, k, n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t blocks = (n + 255) / 256;
  const int64_t cap = (int64_t)cu_count * 4;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  if (n > 0 && k > 0) {
    for (int pass = 0; pass < kPasses; ++pass) {
      hipLaunchKernelGGL(topk_hist, dim3((unsigned)blocks), dim3(256), 0, s, valid, scores, n,
                         st, hist);
      hipLaunchKernelGGL(topk_pick, dim3(1), dim3(256), 0, s, st, hist, pass);
    }
    hipLaunchKernelGGL(topk_gather, dim3((unsigned)blocks), dim3(256), 0, s, valid, scores, n,
                       st, cand);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  int size = 1;
  while (size < k) size <<= 1;
  const size_t lds = (size_t)size * sizeof(unsigned long long);
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(&topk_sort),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(topk_sort, dim3(1), dim3(kSortThreads), lds, s, scores, st, cand, idx,
                     score, num);
  return hipGetLastError();
}

hipError_t launch_rerank_select(const int32_t *rows, const float *scores, int32_t m, int64_t n,
                                int32_t keep, int32_t *idx, float *score, int32_t *num,
                                hipStream_t s) {
  int size = 1;
  while (size < m) size <<= 1;
  const size_t lds = (size_t)size * sizeof(unsigned long long);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&rerank_select),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
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
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&merge_held),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_held, dim3(1), dim3(kSortThreads), lds, s, h_id, h_p, h_a, h_n, c_idx,
                     c_p, c_a, c_n, row0, k, o_id, o_p, o_a, o_n);
  return hipGetLastError();
}

}  // namespace ml2
