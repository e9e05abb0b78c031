// Rule book construction on the GPU (Sec. 3.2.2, Eq. 10; Sec. 3.2.3, the rule-book part of Alg. 1).
//
// Instead of Alg. 1's all-pairs loop, every input site is inserted into an
// open-addressing hash table in HBM (64-bit slots key<<32 | row, lock-free
// atomicCAS, linear probing), and on submanifold layers every (output site, offset) pair
// probes it once for y = stride*x - s (half the offsets; the other half mirrored).
// Results:
//   nbr[s][x]   neighbour map (input row or -1), offset-major so that the
//               forward gather reads one coalesced index vector per offset;
//   pairs       R_s for every offset, compacted with wavefront ballots and a
//               device-wide scan (count pass, scan, write pass), so the order
//               is deterministic: grouped by s, output rows ascending.
// Dilated / strided output sets are marked in a bitmap over the output grid
// and emitted in lexicographic (b, x, y, z) order by a scan of popcounts; their
// neighbour map is written from the input side, the output row of each marked
// (input, offset) being the rank of its bit, so no table of the outputs is
// probed (it is built only if a caller asks for it).
#include <algorithm>
#include <cstdio>
#include <mutex>
#include <vector>

#include "hash.hpp"
#include "scan.hpp"

namespace ssconv {

namespace {

constexpr int kFlagBounds = 1, kFlagDup = 2, kFlagFull = 4;

__global__ void validate_kernel(const int32_t* __restrict__ c, int64_t n, int g0, int g1, int g2,
                                int* __restrict__ flags, int* __restrict__ maxb) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int bad = 0, mb = -1;
  if (i < n) {
    int4 v = reinterpret_cast<const int4*>(c)[i];
    bad = (v.x < 0) | (v.y < 0) | (v.y >= g0) | (v.z < 0) | (v.z >= g1) | (v.w < 0) | (v.w >= g2);
    mb = v.x;
  }
  // one atomic per wavefront
  for (int d = 32; d >= 1; d >>= 1) {
    bad |= __shfl_xor(bad, d, 64);
    mb = max(mb, __shfl_xor(mb, d, 64));
  }
  if ((threadIdx.x & 63) == 0) {
    if (bad) atomicOr(flags, kFlagBounds);
    atomicMax(maxb, mb);
  }
}

// Empty hash slots; the first thread also clears the build flags when asked (flags[0] = 0,
// flags[1] = max batch index seen = -1).
__global__ void fill_slots(uint64_t* __restrict__ p, int64_t n, uint64_t v, int* __restrict__ flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (flags && i == 0) {
    flags[0] = 0;
    flags[1] = -1;
  }
  if (i < n) p[i] = v;
}

// Inserts every site; a site outside the grid, with b < 0 or with b > bmax (the largest batch
// index whose keys fit 32 bits) is not inserted and raises kFlagBounds (one atomic per
// wavefront that holds such a site).
// copy (optional): every coordinate row is also written there (the output sites of a submanifold
// layer are its input sites).
__global__ void hash_insert_kernel(const int32_t* __restrict__ c, int64_t n, int g0, int g1, int g2, int bmax,
                                   uint64_t* __restrict__ slots, uint64_t mask, int* __restrict__ flags,
                                   int32_t* __restrict__ copy) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int4 v = make_int4(0, 0, 0, 0);
  bool bad = false;
  if (i < n) {
    v = reinterpret_cast<const int4*>(c)[i];
    if (copy) reinterpret_cast<int4*>(copy)[i] = v;
    bad = (v.x < 0) | (v.x > bmax) | (v.y < 0) | (v.y >= g0) | (v.z < 0) | (v.z >= g1) | (v.w < 0) | (v.w >= g2);
  }
  const uint64_t any_bad = __ballot(bad);
  if (any_bad && (threadIdx.x & 63) == __ffsll((unsigned long long)any_bad) - 1) atomicOr(flags, kFlagBounds);
  if (i >= n || bad) return;
  uint32_t key = site_key(v.x, v.y, v.z, v.w, g0, g1, g2);
  uint64_t item = ((uint64_t)key << 32) | (uint32_t)i;
  uint64_t pos = mix32(key) & mask;
  for (uint64_t probe = 0; probe <= mask; ++probe) {
    unsigned long long prev =
        atomicCAS(reinterpret_cast<unsigned long long*>(&slots[pos]), (unsigned long long)kEmpty,
                  (unsigned long long)item);
    if (prev == kEmpty) return;
    if ((uint32_t)(prev >> 32) == key) {
      atomicOr(flags, kFlagDup);
      return;
    }
    pos = (pos + 1) & mask;
  }
  atomicOr(flags, kFlagFull);
}

// Output-set marking: for input y and offset s, stride*x = y + s must divide exactly.  Offsets run
// over {-h .. ksize-1-h}^3 with h = ksize/2: {-h..h}^3 for odd kernels, {-1, 0}^3 for the 2x2x2
// pooling windows (y = 2x + {0,1}^3).
__global__ void mark_outputs(const int32_t* __restrict__ c, int64_t n, int ksize, int stride, int go0, int go1,
                             int go2, uint32_t* __restrict__ bits) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int s = blockIdx.y;
  if (i >= n) return;
  int h = ksize / 2;
  int dx = s / (ksize * ksize) - h, dy = (s / ksize) % ksize - h, dz = s % ksize - h;
  int4 v = reinterpret_cast<const int4*>(c)[i];
  int tx = v.y + dx, ty = v.z + dy, tz = v.w + dz;
  if (tx < 0 || ty < 0 || tz < 0) return;
  if (tx % stride || ty % stride || tz % stride) return;
  int x = tx / stride, y = ty / stride, z = tz / stride;
  if (x >= go0 || y >= go1 || z >= go2) return;
  uint64_t bit = (((uint64_t)v.x * go0 + x) * go1 + y) * go2 + z;
  atomicOr(&bits[bit >> 5], 1u << (bit & 31));
}

// One thread per bit of the output bitmap (bit index < 2^32: it is a 32-bit site key): a set bit
// is output row woff[word] + (set bits below it in its word), so the rows come out in
// lexicographic (b, x, y, z) order.
__global__ void emit_outputs(const uint32_t* __restrict__ bits, int64_t nbits, const int64_t* __restrict__ woff,
                             int go0, int go1, int go2, int32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nbits) return;
  const uint32_t bit = (uint32_t)i, b = bit & 31u;
  const uint32_t m = bits[bit >> 5];
  if (!((m >> b) & 1u)) return;
  const int64_t o = woff[bit >> 5] + __popc(m & ((1u << b) - 1u));
  const uint32_t g2 = (uint32_t)go2, g12 = (uint32_t)go1 * g2, per_b = (uint32_t)go0 * g12;
  const uint32_t bb = bit / per_b, r = bit - bb * per_b;
  const uint32_t x = r / g12, yz = r - x * g12;
  const uint32_t y = yz / g2, z = yz - y * g2;
  reinterpret_cast<int4*>(out)[o] = make_int4((int)bb, (int)x, (int)y, (int)z);
}

// Neighbour map of a generated output set, filled from the input side: the marking above already
// names, for input y and offset s, the one output x with stride*x = y + d(s), and that output's
// row is the rank of its bit (as in emit_outputs), so nbr[s][row(x)] = y needs no hash lookup.
// Distinct inputs give distinct (x, s), so every entry is written at most once (duplicate inputs
// fail the build).  nbr is preset to -1.  Grid (ceil(n / 256), K).
__global__ void scatter_neighbours(const int32_t* __restrict__ c, int64_t n, int ksize, int stride, int go0, int go1,
                                   int go2, const uint32_t* __restrict__ bits, const int64_t* __restrict__ woff,
                                   int64_t n_out, int32_t* __restrict__ nbr) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int s = blockIdx.y;
  if (i >= n) return;
  const int h = ksize / 2;
  const int dx = s / (ksize * ksize) - h, dy = (s / ksize) % ksize - h, dz = s % ksize - h;
  const int4 v = reinterpret_cast<const int4*>(c)[i];
  const int tx = v.y + dx, ty = v.z + dy, tz = v.w + dz;
  if (tx < 0 || ty < 0 || tz < 0) return;
  if (tx % stride || ty % stride || tz % stride) return;
  const int x = tx / stride, y = ty / stride, z = tz / stride;
  if (x >= go0 || y >= go1 || z >= go2) return;
  const uint64_t bit = (((uint64_t)v.x * go0 + x) * go1 + y) * go2 + z;
  const uint32_t b = (uint32_t)(bit & 31u), m = bits[bit >> 5];
  const int64_t row = woff[bit >> 5] + __popc(m & ((1u << b) - 1u));
  nbr[(int64_t)s * n_out + row] = (int32_t)i;
}

// Logical (row block, offset) of workgroup blockIdx.x in a 1-D launch of nblk * nS workgroups.
// Workgroup ids are dispatched round-robin over the 8 XCDs (id % 8); each XCD is given one
// contiguous range of logical ids, row block first, so an XCD looks up every offset of a
// contiguous range of sites and the hash lines those lookups touch stay in its own L2.
__device__ __forceinline__ void xcd_tile(int64_t total, int nS, int64_t* rblk, int* s) {
  const int64_t w = blockIdx.x;
  const int x = (int)(w & 7);
  const int64_t q = total >> 3;
  const int r = (int)(total & 7);
  const int64_t L = x * q + min(x, r) + (w >> 3);
  *rblk = L / nS;
  *s = (int)(L - *rblk * nS);
}

__device__ __forceinline__ int lookup(const int32_t* __restrict__ out_c, int64_t p, int s, int ksize, int stride,
                                      int g0, int g1, int g2, const uint64_t* __restrict__ slots, uint64_t mask) {
  const int h = ksize / 2;
  const int dx = s / (ksize * ksize) - h, dy = (s / ksize) % ksize - h, dz = s % ksize - h;
  const int4 v = reinterpret_cast<const int4*>(out_c)[p];
  const int yx = stride * v.y - dx, yy = stride * v.z - dy, yz = stride * v.w - dz;
  if (yx < 0 || yy < 0 || yz < 0 || yx >= g0 || yy >= g1 || yz >= g2) return -1;
  return hash_find(slots, mask, site_key(v.x, yx, yy, yz, g0, g1, g2));
}

// Pair-list passes over (offset s, block of 256 output rows) of a finished neighbour map:
//   kCount  counts the pairs per (offset, block) (grid (nblk, K));
//   kWrite  writes the pairs at the scanned offsets (grid (nblk, K)).
constexpr int kCount = 1, kWrite = 2;
template <int kMode>
__global__ __launch_bounds__(256) void pair_list_kernel(int64_t n_out, int nblk, const int32_t* __restrict__ nbr,
                                                        int32_t* __restrict__ counts, const int64_t* __restrict__ offs,
                                                        int32_t* __restrict__ pairs) {
  __shared__ int wcount[4];
  const int64_t rblk = blockIdx.x;
  const int s = blockIdx.y;
  const int64_t p = rblk * 256 + threadIdx.x;
  const int nb = p < n_out ? nbr[(int64_t)s * n_out + p] : -1;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t ball = __ballot(nb >= 0);
  if (lane == 0) wcount[w] = __popcll(ball);
  __syncthreads();
  if (kMode != kWrite) {
    if (threadIdx.x == 0) counts[(int64_t)s * nblk + rblk] = wcount[0] + wcount[1] + wcount[2] + wcount[3];
  } else if (nb >= 0) {
    int before = 0;
    for (int i = 0; i < w; ++i) before += wcount[i];
    const uint64_t lower = lane ? (ball & ((1ull << lane) - 1)) : 0ull;
    int64_t at = offs[(int64_t)s * nblk + rblk] + before + __popcll(lower);
    reinterpret_cast<int2*>(pairs)[at] = make_int2((int)p, nb);
  }
}

// Tiles of the pair compaction below: kCompactTile consecutive entries of the flattened map.
constexpr int kCompactNT = 256, kCompactPer = 32, kCompactTile = kCompactNT * kCompactPer;
constexpr int kCompactShift = 13;
static_assert(kCompactTile == 1 << kCompactShift, "tile index by shift");

// Adds this wavefront's present entries to the counts of the compaction tiles that hold them
// (f: the entry's index in the flattened map): one atomic per distinct tile of the wavefront.
__device__ __forceinline__ void count_tiles(bool present, int64_t f, int64_t* __restrict__ tile_cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t t = f >> kCompactShift;
  uint64_t left = __ballot(present);
  while (left) {
    const int leader = __ffsll((unsigned long long)left) - 1;
    const int64_t tl = __shfl(t, leader, 64);
    const uint64_t same = __ballot(present && t == tl);
    if (lane == leader) atomicAdd((unsigned long long*)&tile_cnt[tl], (unsigned long long)__popcll(same));
    left &= ~same;
  }
}

// Submanifold layers (one site set, rows shared): only the offsets s < c = (K-1)/2 are looked
// up.  If site x has neighbour y at offset s (y = x - d(s)), then y has neighbour x at the
// mirrored offset K-1-s (d(K-1-s) = -d(s)), so that entry is written from here; distinct x
// give distinct y, so every entry is written at most once.  Rows c..K-1 are set beforehand by
// rb_init_kernel (c: the identity, above c: -1).  Every entry written here is also counted into the
// compaction tile that holds it (tile_cnt, preset by rb_init_kernel with the centre row's entries),
// so the compaction needs no counting pass.  1-D XCD-ordered launch of nblk * c workgroups.
__global__ __launch_bounds__(256) void mirror_lookup_kernel(const int32_t* __restrict__ c_in, int64_t n, int ksize,
                                                            int g0, int g1, int g2,
                                                            const uint64_t* __restrict__ slots, uint64_t mask,
                                                            int nblk, int32_t* __restrict__ nbr,
                                                            int64_t* __restrict__ tile_cnt) {
  const int K = ksize * ksize * ksize, c = (K - 1) / 2;
  int64_t rblk;
  int s;
  xcd_tile((int64_t)nblk * c, c, &rblk, &s);
  const int64_t p = rblk * 256 + threadIdx.x;
  if (p >= n) return;
  const int nb = lookup(c_in, p, s, ksize, 1, g0, g1, g2, slots, mask);
  nbr[(int64_t)s * n + p] = nb;
  if (nb >= 0) nbr[(int64_t)(K - 1 - s) * n + nb] = (int32_t)p;
  count_tiles(nb >= 0, (int64_t)s * n + p, tile_cnt);
  count_tiles(nb >= 0, (int64_t)(K - 1 - s) * n + (nb >= 0 ? nb : 0), tile_cnt);
}

// One launch that prepares a build (thread i handles entry i of every region it reaches):
//   slots[0, cap)            <- empty                         (the hash table)
//   map[0, rows * n)         <- -1, except map[i] = i for i < n when first_identity
//                               (submanifold: rows c..K-1 of the neighbour map, c = centre;
//                               generated sets: the whole map)
//   flags[0] = 0, flags[1] = -1                               (when flags is given)
//   tile_cnt[0, ntiles)      <- the entries [c0, c0 + n) (the centre row) in each compaction tile
//                               (when tile_cnt is given; the lookups add the rest)
__global__ void rb_init_kernel(uint64_t* __restrict__ slots, int64_t cap, int32_t* __restrict__ map, int64_t rows,
                               int64_t n, int first_identity, int* __restrict__ flags,
                               int64_t* __restrict__ tile_cnt = nullptr, int64_t ntiles = 0, int64_t c0 = 0) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cap) slots[i] = kEmpty;
  if (i < rows * n) map[i] = (first_identity && i < n) ? (int32_t)i : -1;
  if (flags && i == 0) {
    flags[0] = 0;
    flags[1] = -1;
  }
  if (tile_cnt && i < ntiles) {
    const int64_t lo = max(i * kCompactTile, c0), hi = min((i + 1) * kCompactTile, c0 + n);
    tile_cnt[i] = hi > lo ? hi - lo : 0;
  }
}

// Compaction of the neighbour map into the pair lists.  The map nbr[K][n] is read as one array in
// its own (offset-major) order, so the pairs come out grouped by offset with output rows
// ascending: pairs[pos] = (row, nbr[s][row]) for every entry >= 0, pos = the number of such
// entries before it; pair_off[s] = the count before offset s's first entry, pair_off[K] = all.
// The array is cut into tiles of kCompactTile entries, one workgroup each; step j of thread t of a
// tile is its entry j * kCompactNT + t (coalesced loads, and the valid lanes of one wavefront
// step write consecutive pairs).  Two launches: pair_count_kernel writes every tile's count,
// pair_write_kernel adds the counts of the tiles before its own (at most a few thousand values,
// read from L2) and writes its pairs.  No workgroup waits on another.  A submanifold build has its
// counts from the lookups already (mirror_lookup_kernel) and skips the counting launch.

// Loads a tile's entries (-1 past the end) and the ballot of valid lanes per step.
__device__ __forceinline__ void compact_load(const int32_t* __restrict__ nbr, int64_t f0, int64_t total, int tid,
                                             int (&v)[kCompactPer], uint64_t (&bal)[kCompactPer]) {
#pragma unroll
  for (int j = 0; j < kCompactPer; ++j) {
    const int64_t f = f0 + (int64_t)j * kCompactNT + tid;
    v[j] = f < total ? nbr[f] : -1;
  }
#pragma unroll
  for (int j = 0; j < kCompactPer; ++j) bal[j] = __ballot(v[j] >= 0);
}

__global__ __launch_bounds__(kCompactNT) void pair_count_kernel(const int32_t* __restrict__ nbr, int64_t total,
                                                                int64_t* __restrict__ tile_count) {
  __shared__ int s_w[kCompactNT / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int v[kCompactPer];
  uint64_t bal[kCompactPer];
  compact_load(nbr, (int64_t)blockIdx.x * kCompactTile, total, tid, v, bal);
  int c = 0;
#pragma unroll
  for (int j = 0; j < kCompactPer; ++j) c += __popcll(bal[j]);
  if (lane == 0) s_w[w] = c;
  __syncthreads();
  if (tid == 0) {
    int64_t t = 0;
    for (int i = 0; i < kCompactNT / 64; ++i) t += s_w[i];
    tile_count[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(kCompactNT) void pair_write_kernel(const int32_t* __restrict__ nbr, int64_t n, int K,
                                                                const int64_t* __restrict__ tile_count,
                                                                int32_t* __restrict__ pairs,
                                                                int64_t* __restrict__ pair_off) {
  constexpr int NW = kCompactNT / 64;
  __shared__ int s_cnt[kCompactPer][NW];  // valid entries per (step, wavefront)
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t tile = blockIdx.x;
  const int64_t total = (int64_t)K * n;
  const int64_t f0 = tile * kCompactTile;
  int v[kCompactPer];
  uint64_t bal[kCompactPer];
  compact_load(nbr, f0, total, tid, v, bal);
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < kCompactPer; ++j) s_cnt[j][w] = __popcll(bal[j]);
  }
  int64_t part = 0;
  for (int64_t i = tid; i < tile; i += kCompactNT) part += tile_count[i];
  int64_t before = 0;
  block_excl_scan<kCompactNT, int64_t>(part, &before);  // also orders the s_cnt writes before the reads
  // this wavefront's position at step 0: every (step, wavefront) count before it in entry order
  int64_t pos = before;
  for (int i = 0; i < w; ++i) pos += s_cnt[0][i];
  const uint64_t below = (1ull << lane) - 1ull;
  int64_t f = f0 + tid;
  int64_t s = f / n, p = f - s * n;
#pragma unroll
  for (int j = 0; j < kCompactPer; ++j) {
    if (f < total) {
      const int64_t at = pos + __popcll(bal[j] & below);
      if (p == 0) pair_off[s] = at;
      if (v[j] >= 0) reinterpret_cast<int2*>(pairs)[at] = make_int2((int)p, v[j]);
    }
    // to step j + 1: the rest of this step (wavefronts from w on) and the next step's wavefronts before w
    if (j + 1 < kCompactPer) {
#pragma unroll
      for (int i = 0; i < NW; ++i) pos += (i >= w ? s_cnt[j][i] : 0) + (i < w ? s_cnt[j + 1][i] : 0);
      f += kCompactNT;
      if (f < total) {
        if (n < kCompactNT) {
          s = f / n, p = f - s * n;
        } else if ((p += kCompactNT) >= n) {  // p + kCompactNT < 2n
          p -= n, ++s;
        }
      }
    }
  }
  if (tile == gridDim.x - 1 && tid == 0) {
    int64_t all = before;
    for (int i = 0; i < kCompactPer * NW; ++i) all += s_cnt[i / NW][i % NW];
    pair_off[K] = all;
  }
}

// The launches of the compaction; tile_count holds compact_tiles(K, n) values, already the counts
// when counted.
int compact_pairs(const int32_t* nbr, int64_t n, int K, int64_t* tile_count, int32_t* pairs, int64_t* pair_off,
                  hipStream_t st, bool counted = false);

int64_t compact_tiles(int64_t K, int64_t n) { return (K * n + kCompactTile - 1) / kCompactTile; }

int compact_pairs(const int32_t* nbr, int64_t n, int K, int64_t* tile_count, int32_t* pairs, int64_t* pair_off,
                  hipStream_t st, bool counted) {
  const int64_t tiles = compact_tiles(K, n);
  if (!counted) pair_count_kernel<<<(unsigned)tiles, kCompactNT, 0, st>>>(nbr, (int64_t)K * n, tile_count);
  pair_write_kernel<<<(unsigned)tiles, kCompactNT, 0, st>>>(nbr, n, K, tile_count, pairs, pair_off);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int64_t next_pow2(int64_t v) {
  int64_t c = 64;
  while (c < v) c <<= 1;
  return c;
}

// Pinned host staging for the few values the build reads back.
struct Staging {
  int64_t* p = nullptr;
  int get(int64_t** out) {
    if (!p) {
      void* q = nullptr;
      if (hipHostMalloc(&q, 4096, hipHostMallocDefault) != hipSuccess || !q) {
        (void)hipGetLastError();
        return fail(SSCONV_E_NOMEM, "pinned host staging allocation failed");
      }
      p = (int64_t*)q;
    }
    *out = p;
    return SSCONV_OK;
  }
};
thread_local Staging g_stage;

// Pinned read-back buffers and events of asynchronous builds, reused across builds (a pinned
// allocation or an event creation per build would cost host time on every call).
struct StagePool {
  std::mutex mu;
  std::vector<std::pair<int64_t*, hipEvent_t>> free_list;
  int get(int64_t** buf, hipEvent_t* ev) {
    {
      std::lock_guard<std::mutex> lk(mu);
      if (!free_list.empty()) {
        *buf = free_list.back().first;
        *ev = free_list.back().second;
        free_list.pop_back();
        return SSCONV_OK;
      }
    }
    void* q = nullptr;
    if (hipHostMalloc(&q, 4096, hipHostMallocDefault) != hipSuccess || !q) {
      (void)hipGetLastError();
      return fail(SSCONV_E_NOMEM, "pinned host staging allocation failed");
    }
    if (hipEventCreateWithFlags(ev, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipHostFree(q);
      return fail(SSCONV_E_HIP, "event creation failed");
    }
    *buf = (int64_t*)q;
    return SSCONV_OK;
  }
  void put(int64_t* buf, hipEvent_t ev) {
    std::lock_guard<std::mutex> lk(mu);
    free_list.emplace_back(buf, ev);
  }
};
StagePool g_stage_pool;

// Reads the pair counts and the build flags from host memory (the read-back has completed).
int settle_from(ssconv_rulebook* rb, const int64_t* host) {
  const int K = rb->K;
  for (int s = 0; s <= K; ++s) rb->pair_off[s] = host[s];
  rb->n_pairs = host[K];
  const int fl = (int)(host[K + 1] & 0xffffffff);
  if (fl & kFlagBounds) return fail(SSCONV_E_BOUNDS, "a site lies outside the grid, has b < 0, or (max b + 1) * grid volume exceeds the 32-bit key space");
  if (fl & kFlagDup) return fail(SSCONV_E_DUPLICATE, "duplicate input site");
  if (fl & kFlagFull) return fail(SSCONV_E_HASH_FULL, "coordinate hash table is full");
  return SSCONV_OK;
}

}  // namespace

int rulebook_settle(ssconv_rulebook* rb) {
  if (rb->pending) {
    rb->pending = false;
    int rc;
    if (hipEventSynchronize(rb->ready) != hipSuccess) {
      (void)hipGetLastError();
      rc = fail(SSCONV_E_HIP, "waiting for the rule book build failed");
    } else {
      rc = settle_from(rb, rb->stage);
    }
    rb->status = rc;
    if (rc != SSCONV_OK) snprintf(rb->error, sizeof(rb->error), "%s", ssconv_last_error());
    return rc;
  }
  if (rb->status != SSCONV_OK) return fail(rb->status, "%s", rb->error);
  return SSCONV_OK;
}

void rulebook_free(ssconv_rulebook* rb) {
  if (!rb) return;
  if (rb->stage) {
    if (rb->pending) (void)hipEventSynchronize(rb->ready);  // the read-back still writes the stage
    (void)hipGetLastError();
    g_stage_pool.put(rb->stage, rb->ready);
  }
  for (void* m : rb->mem) dev_free(m, rb->stream);  // every device buffer lives in these blocks
  delete[] rb->pair_off;
  delete rb;
}

// Carves 256-byte aligned pieces out of one allocation.
struct Carve {
  size_t at = 0;
  size_t take(size_t bytes) {
    const size_t o = at;
    at += (bytes + 255) & ~(size_t)255;
    return o;
  }
};

// Temporary device buffers released on every exit path.
struct Scratch {
  hipStream_t s;
  void* ptrs[8] = {};
  int n = 0;
  explicit Scratch(hipStream_t st) : s(st) {}
  int alloc(void** p, size_t bytes) {
    SSC_TRY(dev_alloc(p, bytes, s));
    ptrs[n++] = *p;
    return SSCONV_OK;
  }
  ~Scratch() {
    for (int i = 0; i < n; ++i) dev_free(ptrs[i], s);
  }
};

// largest batch index whose site keys ((b*G0 + x)*G1 + y)*G2 + z fit in 32 bits (key ~0 is reserved)
static int max_batch(const int* g) {
  const int64_t cells = (int64_t)g[0] * g[1] * g[2];
  const int64_t m = 0xFFFFFFFFll / cells - 1;
  return (int)std::min<int64_t>(m, 0x7fffffff);
}

static int hash_capacity(int64_t n, int64_t* cap) {
  int64_t c = debug_hash_capacity();
  if (c <= 0) c = next_pow2(2 * n);
  if (c & (c - 1)) return fail(SSCONV_E_INVALID, "forced hash capacity must be a power of two");
  *cap = c;
  return SSCONV_OK;
}

// Fills the table (capacity cap, already allocated) and inserts the n sites; init_flags also
// clears the build flags in the fill kernel, validate also records the largest batch index in
// flags[1] (and bounds violations in flags[0]) before the inserts.
static int build_hash(const int32_t* coords, int64_t n, const int* g, hipStream_t st, uint64_t* slots, int64_t cap,
                      int* flags, bool init_flags, bool validate) {
  fill_slots<<<cdiv(cap, 256), 256, 0, st>>>(slots, cap, kEmpty, init_flags ? flags : nullptr);
  if (validate && n > 0) validate_kernel<<<cdiv(n, 256), 256, 0, st>>>(coords, n, g[0], g[1], g[2], flags, flags + 1);
  if (n > 0)
    hash_insert_kernel<<<cdiv(n, 256), 256, 0, st>>>(coords, n, g[0], g[1], g[2], max_batch(g), slots,
                                                     (uint64_t)(cap - 1), flags, nullptr);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

// Pair offsets and flags in one copy: the one synchronisation of a submanifold build (the last of
// a generated one); device-detected errors surface here.
// The one read-back of a build: the pair counts and the flags.  async: queued into a pooled
// pinned buffer with an event behind it, settled later (rulebook_settle).
static int finish_build(ssconv_rulebook* rb, int64_t* host, hipStream_t st, bool async) {
  const int K = rb->K;
  if (async) {
    SSC_TRY(g_stage_pool.get(&rb->stage, &rb->ready));
    SSC_HIP(hipMemcpyAsync(rb->stage, rb->pair_off_dev, (size_t)(K + 2) * 8, hipMemcpyDeviceToHost, st));
    SSC_HIP(hipEventRecord(rb->ready, st));
    rb->pending = true;
    return SSCONV_OK;
  }
  SSC_HIP(hipMemcpyAsync(host, rb->pair_off_dev, (size_t)(K + 2) * 8, hipMemcpyDeviceToHost, st));
  SSC_HIP(hipStreamSynchronize(st));
  return settle_from(rb, host);
}

static int build_impl(const int32_t* coords, int64_t n, const int32_t* grid, int ksize, int stride, int submanifold,
                      hipStream_t st, ssconv_rulebook* rb, bool async) {
  rb->ksize = ksize;
  rb->K = ksize * ksize * ksize;
  rb->stride = stride;
  rb->submanifold = submanifold;
  rb->stream = st;
  rb->n_in = n;
  for (int a = 0; a < 3; ++a) {
    rb->grid[a] = grid[a];
    rb->grid_out[a] = (grid[a] + stride - 1) / stride;
  }
  const int K = rb->K;
  rb->pair_off = new int64_t[K + 1]();
  int64_t* host = nullptr;
  SSC_TRY(g_stage.get(&host));
  // Device memory comes in few allocations (each costs host time on every build): the handle's
  // buffers in at most three blocks, the temporaries in one or two.  pair_off_dev is followed by
  // the build flags, so both come back in one copy.
  SSC_TRY(hash_capacity(n, &rb->cap_in));
  const size_t pairs_bound = (size_t)K * (size_t)n * 8;  // submanifold: every output has <= K pairs
  const bool pairs_in_block = submanifold && pairs_bound <= ((size_t)1 << 30);
  int* dflags = nullptr;  // [0] flags, [1] max b
  int64_t* tile_cnt = nullptr;  // per-tile counts of the pair compaction (submanifold builds)
  const int64_t sub_tiles = submanifold ? compact_tiles(K, n) : 0;
  {
    Carve c;
    const size_t o_hash = c.take((size_t)rb->cap_in * 8), o_off = c.take((size_t)(K + 2) * 8);
    size_t o_oc = 0, o_nbr = 0, o_pairs = 0, o_lb = 0;
    if (submanifold) {
      o_oc = c.take((size_t)n * 16);
      o_nbr = c.take((size_t)K * n * 4);
      if (pairs_in_block) o_pairs = c.take(pairs_bound);
      o_lb = c.take((size_t)sub_tiles * 8);
    }
    char* b0 = nullptr;
    SSC_TRY(dev_alloc((void**)&b0, c.at, st));
    rb->mem[0] = b0;
    rb->hash_in = (uint64_t*)(b0 + o_hash);
    rb->pair_off_dev = (int64_t*)(b0 + o_off);
    dflags = (int*)(rb->pair_off_dev + K + 1);
    if (submanifold) {
      rb->out_coords = (int32_t*)(b0 + o_oc);
      rb->nbr = (int32_t*)(b0 + o_nbr);
      if (pairs_in_block) rb->pairs = (int32_t*)(b0 + o_pairs);
      tile_cnt = (int64_t*)(b0 + o_lb);
    }
  }

  if (submanifold && n > 0) {
    // Four launches and one read-back: (1) the table, the mirrored rows of the neighbour map, the
    // compaction's tile counts (the centre row's share) and the flags are set by one kernel; (2) the
    // inserts, which also copy the sites (the output set); (3) lookups of the offsets before the
    // centre, mirrored entries written from them, every entry counted into its compaction tile;
    // (4) the single-pass compaction into the pair lists.
    const int c = (K - 1) / 2;
    const int64_t init_n0 = std::max<int64_t>(rb->cap_in, (int64_t)(K - c) * n);
    rb->n_out = n;
    rb->hash_out = rb->hash_in;
    rb->cap_out = rb->cap_in;
    const int64_t init_n = std::max<int64_t>(init_n0, sub_tiles);
    rb_init_kernel<<<cdiv(init_n, 256), 256, 0, st>>>(rb->hash_in, rb->cap_in, rb->nbr + (int64_t)c * n, K - c, n, 1,
                                                      dflags, tile_cnt, sub_tiles, (int64_t)c * n);
    hash_insert_kernel<<<cdiv(n, 256), 256, 0, st>>>(coords, n, grid[0], grid[1], grid[2], max_batch(rb->grid),
                                                     rb->hash_in, (uint64_t)(rb->cap_in - 1), dflags, rb->out_coords);
    const int nblk = (int)cdiv(n, 256);
    if (c > 0)
      mirror_lookup_kernel<<<(unsigned)((int64_t)nblk * c), 256, 0, st>>>(rb->out_coords, n, ksize, grid[0], grid[1],
                                                                          grid[2], rb->hash_in,
                                                                          (uint64_t)(rb->cap_in - 1), nblk, rb->nbr,
                                                                          tile_cnt);
    SSC_HIP(hipGetLastError());
    if (rb->pairs) {
      SSC_TRY(compact_pairs(rb->nbr, n, K, tile_cnt, rb->pairs, rb->pair_off_dev, st, true));
      return finish_build(rb, host, st, async);
    }
    // past 1 GB of pairs at the upper bound: counted, scanned and sized exactly below
  }

  // the input table's fill also clears the build flags; its inserts do not depend on the output
  // set, so for generated sets they are queued before the synchronisation that sizes the bitmap
  if (!(submanifold && n > 0))
    SSC_TRY(build_hash(coords, n, rb->grid, st, rb->hash_in, rb->cap_in, dflags, true, !submanifold));
  if (!submanifold) {
    // the output bitmap spans the batch: its extent is needed on the host before the next launch
    SSC_HIP(hipMemcpyAsync(host, dflags, 8, hipMemcpyDeviceToHost, st));
    SSC_HIP(hipStreamSynchronize(st));
    const int flags0 = ((int*)host)[0], maxb = ((int*)host)[1];
    if (flags0 & kFlagBounds) return fail(SSCONV_E_BOUNDS, "a site lies outside the grid, has b < 0, or (max b + 1) * grid volume exceeds the 32-bit key space");
    if (maxb > max_batch(grid)) return fail(SSCONV_E_BOUNDS, "(max b + 1) * grid volume exceeds the 32-bit key space");
    // no valid rule book follows a duplicate site or a full table: the build ends here, before the
    // output set and the map are built
    if (flags0 & kFlagDup) return fail(SSCONV_E_DUPLICATE, "duplicate input site");
    if (flags0 & kFlagFull) return fail(SSCONV_E_HASH_FULL, "coordinate hash table is full");
    rb->nbatch = maxb + 1;
  }

  // ---- output site set ----
  Scratch tmp(st);
  uint32_t* obits = nullptr;  // generated sets: output bitmap and its word offsets (ranks)
  int64_t* owoff = nullptr;
  if (submanifold) {
    rb->n_out = n;  // sites copied and the map's mirrored rows set above
    rb->hash_out = rb->hash_in;
    rb->cap_out = rb->cap_in;
  } else {
    const int* go = rb->grid_out;
    const int64_t nbits = rb->nbatch * (int64_t)go[0] * go[1] * go[2];
    const int64_t nw = (nbits + 31) / 32;
    Carve c;
    const size_t o_bits = c.take((size_t)nw * 4), o_woff = c.take((size_t)nw * 8),
                 o_stmp = c.take((size_t)scan_tmp_elems(nw) * 8 + 8);
    char* t0 = nullptr;
    SSC_TRY(tmp.alloc((void**)&t0, c.at));
    uint32_t* bits = (uint32_t*)(t0 + o_bits);
    int64_t* woff = (int64_t*)(t0 + o_woff);
    int64_t* stmp = (int64_t*)(t0 + o_stmp);
    int64_t* dtotal = stmp + scan_tmp_elems(nw);
    obits = bits;
    owoff = woff;
    if (nw) SSC_HIP(hipMemsetAsync(bits, 0, (size_t)nw * 4, st));
    if (n > 0) {
      dim3 gm(cdiv(n, 256), K);
      mark_outputs<<<gm, 256, 0, st>>>(coords, n, ksize, stride, go[0], go[1], go[2], bits);
    }
    if (nw) {
      SSC_TRY(exclusive_scan_popc(bits, nw, woff, dtotal, stmp, st));
    } else {
      SSC_HIP(hipMemsetAsync(dtotal, 0, 8, st));
    }
    SSC_HIP(hipMemcpyAsync(host, dtotal, 8, hipMemcpyDeviceToHost, st));
    SSC_HIP(hipStreamSynchronize(st));
    rb->n_out = host[0];
    // second block: output coordinates, output hash (filled only when a caller asks for it: the
    // neighbour map below does not use it), neighbour map, pairs (upper bound <= 1 GB)
    SSC_TRY(hash_capacity(rb->n_out, &rb->cap_out));
    const size_t bound = (size_t)K * (size_t)rb->n_out * 8;
    Carve c1;
    const size_t o_oc = c1.take((size_t)rb->n_out * 16), o_hash = c1.take((size_t)rb->cap_out * 8),
                 o_nbr = c1.take((size_t)K * rb->n_out * 4);
    const size_t o_pairs = bound <= ((size_t)1 << 30) ? c1.take(bound) : 0;
    char* b1 = nullptr;
    SSC_TRY(dev_alloc((void**)&b1, c1.at, st));
    rb->mem[1] = b1;
    rb->out_coords = (int32_t*)(b1 + o_oc);
    rb->hash_out = (uint64_t*)(b1 + o_hash);
    rb->nbr = (int32_t*)(b1 + o_nbr);
    if (bound <= ((size_t)1 << 30)) rb->pairs = (int32_t*)(b1 + o_pairs);
    if (nbits) emit_outputs<<<cdiv(nbits, 256), 256, 0, st>>>(bits, nbits, woff, go[0], go[1], go[2], rb->out_coords);
    SSC_HIP(hipGetLastError());
  }

  // ---- neighbour map and per-offset pair lists ----
  const int64_t n_out = rb->n_out;
  if (n_out > 0) {
    const int nblk = (int)cdiv(n_out, 256);
    const int64_t ncnt = (int64_t)K * nblk;
    Carve c;
    const size_t o_cnt = c.take((size_t)ncnt * 4), o_offs = c.take((size_t)ncnt * 8),
                 o_stmp = c.take((size_t)scan_tmp_elems(ncnt) * 8 + 8),
                 o_lb = c.take((size_t)compact_tiles(K, n_out) * 8);
    char* t1 = nullptr;
    SSC_TRY(tmp.alloc((void**)&t1, c.at));
    int32_t* counts = (int32_t*)(t1 + o_cnt);
    int64_t* offs = (int64_t*)(t1 + o_offs);
    int64_t* stmp = (int64_t*)(t1 + o_stmp);
    int64_t* dtotal = stmp + scan_tmp_elems(ncnt);
    dim3 gp(nblk, K);
    if (submanifold) {
      // the map is complete (set above); only its pair lists are still to be sized and written
      pair_list_kernel<kCount><<<gp, 256, 0, st>>>(n_out, nblk, rb->nbr, counts, nullptr, nullptr);
    } else {
      rb_init_kernel<<<cdiv((int64_t)K * n_out, 256), 256, 0, st>>>(nullptr, 0, rb->nbr, K, n_out, 0, nullptr);
      const int* go = rb->grid_out;
      scatter_neighbours<<<dim3(cdiv(n, 256), K), 256, 0, st>>>(coords, n, ksize, stride, go[0], go[1], go[2], obits,
                                                              owoff, n_out, rb->nbr);
      if (rb->pairs) {
        SSC_TRY(compact_pairs(rb->nbr, n_out, K, (int64_t*)(t1 + o_lb), rb->pairs, rb->pair_off_dev, st));
        return finish_build(rb, host, st, false);
      }
      pair_list_kernel<kCount><<<gp, 256, 0, st>>>(n_out, nblk, rb->nbr, counts, nullptr, nullptr);
    }
    SSC_HIP(hipGetLastError());
    SSC_TRY(exclusive_scan_pair_off(counts, K, nblk, offs, dtotal, stmp, rb->pair_off_dev, st));
    // the pair lists are written at their upper bound (every output has at most K neighbours), so
    // the write pass follows without a round trip to the host and the counts come back once,
    // below; past 1 GB the exact size is read back first
    if (!rb->pairs) {
      SSC_HIP(hipMemcpyAsync(host, dtotal, 8, hipMemcpyDeviceToHost, st));
      SSC_HIP(hipStreamSynchronize(st));
      SSC_TRY(dev_alloc((void**)&rb->mem[2], (size_t)host[0] * 8, st));
      rb->pairs = (int32_t*)rb->mem[2];
    }
    pair_list_kernel<kWrite><<<gp, 256, 0, st>>>(n_out, nblk, rb->nbr, nullptr, offs, rb->pairs);
    SSC_HIP(hipGetLastError());
  } else {
    SSC_HIP(hipMemsetAsync(rb->pair_off_dev, 0, (size_t)(K + 1) * 8, st));
    if (!rb->pairs) {
      SSC_TRY(dev_alloc((void**)&rb->mem[2], 8, st));
      rb->pairs = (int32_t*)rb->mem[2];
    }
  }
  return finish_build(rb, host, st, false);
}

}  // namespace ssconv

using namespace ssconv;

namespace {

int build_entry(const int32_t* coords, int64_t n, const int32_t* grid, int ksize, int stride, int submanifold,
                hipStream_t stream, ssconv_rulebook_t* out, bool async) {
  if (!out) return fail(SSCONV_E_INVALID, "out handle pointer is NULL");
  *out = nullptr;
  if (!grid) return fail(SSCONV_E_INVALID, "grid is NULL");
  if (n < 0 || (n > 0 && !coords)) return fail(SSCONV_E_INVALID, "bad coords/n");
  if (n > 0x7fffffffll) return fail(SSCONV_E_INVALID, "at most 2^31-1 sites");
  if (n > 0 && !aligned16(coords)) return fail(SSCONV_E_INVALID, "coords must be 16-byte aligned");
  if (stride != 1 && stride != 2) return fail(SSCONV_E_INVALID, "stride must be 1 or 2");
  if (submanifold && stride != 1) return fail(SSCONV_E_INVALID, "submanifold requires stride 1");
  if (ksize == 2) {
    if (stride != 2) return fail(SSCONV_E_INVALID, "ksize 2 (pooling windows) requires stride 2, not submanifold");
  } else if (ksize < 1 || ksize > 5 || (ksize & 1) == 0) {
    return fail(SSCONV_E_INVALID, "ksize must be odd, 1..5, or 2 with stride 2");
  }
  for (int a = 0; a < 3; ++a)
    if (grid[a] < 1) return fail(SSCONV_E_INVALID, "grid extents must be positive");
  auto* rb = new ssconv_rulebook();
  int rc = build_impl(coords, n, grid, ksize, stride, submanifold ? 1 : 0, stream, rb, async);
  if (rc != SSCONV_OK) {
    std::string msg = ssconv_last_error();
    rulebook_free(rb);
    set_error("%s", msg.c_str());
    return rc;
  }
  *out = rb;
  return SSCONV_OK;
}

}  // namespace

extern "C" int ssconv_build_rulebook(const int32_t* coords, int64_t n, const int32_t* grid, int ksize, int stride,
                                     int submanifold, hipStream_t stream, ssconv_rulebook_t* out) {
  return build_entry(coords, n, grid, ksize, stride, submanifold, stream, out, false);
}

extern "C" int ssconv_build_rulebook_async(const int32_t* coords, int64_t n, const int32_t* grid, int ksize,
                                           int stride, int submanifold, hipStream_t stream, ssconv_rulebook_t* out) {
  return build_entry(coords, n, grid, ksize, stride, submanifold, stream, out, true);
}

extern "C" int ssconv_rulebook_wait(ssconv_rulebook_t rb) {
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  return rulebook_settle(rb);
}

extern "C" int ssconv_rulebook_info(ssconv_rulebook_t rb, int64_t* n_in, int64_t* n_out, int64_t* pair_counts) {
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  SSC_TRY(rulebook_settle(rb));
  if (n_in) *n_in = rb->n_in;
  if (n_out) *n_out = rb->n_out;
  if (pair_counts)
    for (int s = 0; s < rb->K; ++s) pair_counts[s] = rb->pair_off[s + 1] - rb->pair_off[s];
  return SSCONV_OK;
}

extern "C" int ssconv_rulebook_out_coords(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream) {
  if (!rb || (!dst && rb->n_out)) return fail(SSCONV_E_INVALID, "NULL argument");
  if (rb->n_out) SSC_HIP(hipMemcpyAsync(dst, rb->out_coords, (size_t)rb->n_out * 16, hipMemcpyDeviceToDevice, stream));
  return SSCONV_OK;
}

extern "C" int ssconv_rulebook_pairs(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream) {
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  SSC_TRY(rulebook_settle(rb));
  if (!dst && rb->n_pairs) return fail(SSCONV_E_INVALID, "NULL argument");
  if (rb->n_pairs) SSC_HIP(hipMemcpyAsync(dst, rb->pairs, (size_t)rb->n_pairs * 8, hipMemcpyDeviceToDevice, stream));
  return SSCONV_OK;
}

extern "C" int ssconv_rulebook_neighbours(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream) {
  if (!rb || (!dst && rb->n_out)) return fail(SSCONV_E_INVALID, "NULL argument");
  if (rb->n_out)
    SSC_HIP(hipMemcpyAsync(dst, rb->nbr, (size_t)rb->K * rb->n_out * 4, hipMemcpyDeviceToDevice, stream));
  return SSCONV_OK;
}

extern "C" int ssconv_rulebook_hash(ssconv_rulebook_t rb, int which, uint64_t* dst, int64_t* capacity,
                                    hipStream_t stream) {
  if (!rb || (which != 0 && which != 1)) return fail(SSCONV_E_INVALID, "bad argument");
  SSC_TRY(rulebook_settle(rb));
  if (which && rb->hash_out != rb->hash_in && !rb->hash_out_built) {
    // a generated output set's table is filled on first request, on the caller's stream
    int* dflags = (int*)(rb->pair_off_dev + rb->K + 1);
    SSC_TRY(build_hash(rb->out_coords, rb->n_out, rb->grid_out, stream, rb->hash_out, rb->cap_out, dflags, true, false));
    int flags = 0;
    SSC_HIP(hipMemcpyAsync(&flags, dflags, 4, hipMemcpyDeviceToHost, stream));
    SSC_HIP(hipStreamSynchronize(stream));
    if (flags & kFlagFull) return fail(SSCONV_E_HASH_FULL, "coordinate hash table is full");
    rb->hash_out_built = true;
  }
  const uint64_t* src = which ? rb->hash_out : rb->hash_in;
  int64_t cap = which ? rb->cap_out : rb->cap_in;
  if (capacity) *capacity = cap;
  if (dst) SSC_HIP(hipMemcpyAsync(dst, src, (size_t)cap * 8, hipMemcpyDeviceToDevice, stream));
  return SSCONV_OK;
}

extern "C" void ssconv_rulebook_destroy(ssconv_rulebook_t rb) { rulebook_free(rb); }
