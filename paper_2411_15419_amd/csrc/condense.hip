// luffy_condense: per-bucket cosine threshold graph, representative
// selection and compaction.
//
// Kernels, in launch order:
//   norm_kernel          1/|x_t| per token (one wave per row).
//   gram_prep_kernel     per-bucket tile counts and bitmask offsets.
//   gram_kernel_{bf16,f32}  persistent loop over the upper-triangle 128x128
//                        tiles of every bucket's Gram matrix.  The epilogue
//                        turns cos >= h into adjacency bits and writes both
//                        the tile and its transpose, so every bitmask word is
//                        written exactly once.
//   degree_kernel        popcount of every adjacency row.
//   greedy_round_kernel  one round of the parallel form of the greedy walk
//                        (run a fixed number of times over the whole grid).
//   greedy_finish_kernel one workgroup per bucket repeats rounds until the
//                        bucket is fully decided.
//   assign_kernel        every absorbed position picks its first-visited
//                        adjacent representative.
//   rep_scan_kernel      one workgroup: exclusive scan of the representative
//                        flags -> rows, rep_token, rep_offsets.
//   rep_row_kernel, gather_kernel
//
// The walk of Sec. 5.2 visits positions by priority (degree descending,
// position ascending) and keeps a position iff no neighbour of higher
// priority was kept.  In parallel: an undecided position whose kept
// neighbour exists is absorbed; one whose every higher-priority neighbour is
// absorbed is kept.  Both rules only read final decisions, so rounds may see
// each other's updates early without changing the result, and every round
// decides at least the highest-priority undecided position.
#include "gemm_core.h"
#include "luffy_common.h"

namespace luffy {
namespace {

constexpr int kGreedyGridRounds = 4;
constexpr int kStateUndecided = 0, kStateKept = 1, kStateAbsorbed = 2;

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// first e with offsets[e] <= p < offsets[e+1]
__device__ __forceinline__ int bucket_of(const int32_t* __restrict__ offsets, int E, int p) {
  int lo = 0, hi = E;  // answer: (first i in [0,E] with offsets[i] > p) - 1
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (offsets[mid + 1] <= p) lo = mid + 1; else hi = mid;
  }
  return lo;
}

template <bool BF16>
__global__ __launch_bounds__(256) void norm_kernel(const void* __restrict__ xv, int T, int d,
                                                   float* __restrict__ inv_norm) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  float s = 0.f;
  if constexpr (BF16) {
    const uint16_t* x = static_cast<const uint16_t*>(xv) + static_cast<size_t>(t) * d;
    for (int c = lane * 8; c < d; c += 512) {
      Pack16 v;
      v.u4 = *reinterpret_cast<const uint4*>(x + c);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float f = bf16_to_f32(v.h[i]);
        s = fmaf(f, f, s);
      }
    }
  } else {
    const float* x = static_cast<const float*>(xv) + static_cast<size_t>(t) * d;
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(x + c);
      s = fmaf(v.x, v.x, s);
      s = fmaf(v.y, v.y, s);
      s = fmaf(v.z, v.z, s);
      s = fmaf(v.w, v.w, s);
    }
  }
  s = wave_sum_f32(s);
  if (lane == 0) inv_norm[t] = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
}

// Tile and bitmask layout of every bucket.  Flags an error (and schedules no
// tile) when a bucket exceeds max_bucket or the bitmask exceeds the
// workspace.
__global__ void gram_prep_kernel(const int32_t* __restrict__ offsets, int E, int max_bucket,
                                 long long cap_words, int32_t* __restrict__ tile_off,
                                 long long* __restrict__ bm_off, int* __restrict__ err) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  long long words = 0;
  int tiles = 0, bad = 0;
  for (int e = 0; e < E; ++e) {
    const int n = offsets[e + 1] - offsets[e];
    if (n < 0 || n > max_bucket) bad = 1;
    const int nt = (n + kTile - 1) / kTile;
    tile_off[e] = tiles;
    bm_off[e] = words;
    tiles += nt * (nt + 1) / 2;
    words += static_cast<long long>(n) * ((n + 63) / 64);
  }
  tile_off[E] = tiles;
  bm_off[E] = words;
  if (words > cap_words) bad = 1;
  if (bad)
    for (int e = 0; e <= E; ++e) tile_off[e] = 0;
  *err = bad;
}

struct TileCoord {
  int e, ti, tj, lo, n, W;
};

__device__ __forceinline__ TileCoord decode_tile(int tile, const int32_t* __restrict__ tile_off,
                                                 const int32_t* __restrict__ offsets, int E) {
  TileCoord c;
  int e = 0;
  while (e + 1 < E && tile_off[e + 1] <= tile) ++e;
  const int q = tile - tile_off[e];
  int tj = static_cast<int>((sqrtf(8.0f * q + 1.0f) - 1.0f) * 0.5f);
  while (tj * (tj + 1) / 2 > q) --tj;
  while ((tj + 1) * (tj + 2) / 2 <= q) ++tj;
  c.e = e;
  c.tj = tj;
  c.ti = q - tj * (tj + 1) / 2;
  c.lo = offsets[e];
  c.n = offsets[e + 1] - c.lo;
  c.W = (c.n + 63) / 64;
  return c;
}

// Writes the tile's adjacency words: rows of tile-row ti at words 2tj, 2tj+1
// (from dbits) and, off the diagonal, rows of tile-row tj at words 2ti, 2ti+1
// (from tbits).  dbits/tbits: [128 rows][8 groups of 16 columns].
__device__ __forceinline__ void write_tile_words(const TileCoord& c, const uint16_t (*dbits)[8],
                                                 const uint16_t (*tbits)[8],
                                                 uint64_t* __restrict__ bitmask, long long base) {
  const int tid = threadIdx.x;
  const int rl = tid >> 1, ww = tid & 1;
  auto pack = [](const uint16_t* g) {
    return static_cast<uint64_t>(g[0]) | (static_cast<uint64_t>(g[1]) << 16) |
           (static_cast<uint64_t>(g[2]) << 32) | (static_cast<uint64_t>(g[3]) << 48);
  };
  {
    const int a = c.ti * kTile + rl;
    const int wd = 2 * c.tj + ww;
    if (a < c.n && wd < c.W)
      bitmask[base + static_cast<long long>(a) * c.W + wd] = pack(&dbits[rl][4 * ww]);
  }
  if (c.ti != c.tj) {
    const int b = c.tj * kTile + rl;
    const int wd = 2 * c.ti + ww;
    if (b < c.n && wd < c.W)
      bitmask[base + static_cast<long long>(b) * c.W + wd] = pack(&tbits[rl][4 * ww]);
  }
}

__global__ __launch_bounds__(256, 2) void gram_kernel_bf16(
    const uint16_t* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, float h,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask) {
  __shared__ uint16_t lds[kTileLdsElems];
  __shared__ uint16_t dbits[kTile][8];
  __shared__ uint16_t tbits[kTile][8];
  __shared__ float inv_a[kTile], inv_b[kTile];
  if (*err) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int total = tile_off[E];
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const TileCoord c = decode_tile(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    const uint16_t* prow[4];
    const uint16_t* qrow[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = (tid >> 3) + 32 * q;
      const int a = min(c.ti * kTile + r, c.n - 1);
      const int b = min(c.tj * kTile + r, c.n - 1);
      prow[q] = X + static_cast<size_t>(pt[a]) * d;
      qrow[q] = X + static_cast<size_t>(pt[b]) * d;
    }
    if (tid < kTile) inv_a[tid] = inv_norm[pt[min(c.ti * kTile + tid, c.n - 1)]];
    else inv_b[tid - kTile] = inv_norm[pt[min(c.tj * kTile + tid - kTile, c.n - 1)]];
    reinterpret_cast<uint32_t*>(&dbits[0][0])[tid] = 0u;
    reinterpret_cast<uint32_t*>(&dbits[0][0])[tid + 256] = 0u;
    reinterpret_cast<uint32_t*>(&tbits[0][0])[tid] = 0u;
    reinterpret_cast<uint32_t*>(&tbits[0][0])[tid + 256] = 0u;
    f32x4 acc[4][4];
    zero_acc(acc);
    gemm_tile_bf16(prow, qrow, d, lds, acc);  // ends with a barrier

#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint64_t m[4];
        const int bl = 64 * wn + 16 * j + (lane & 15);
        const int b = c.tj * kTile + bl;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int al = 64 * wm + 16 * i + 4 * (lane >> 4) + r;
          const int a = c.ti * kTile + al;
          const float cs = acc[i][j][r] * inv_a[al] * inv_b[bl];
          m[r] = __ballot(a < c.n && b < c.n && a != b && cs >= h);
        }
        if (m[0] | m[1] | m[2] | m[3]) {
          if (lane < 4) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              dbits[64 * wm + 16 * i + 4 * lane + r][4 * wn + j] =
                  static_cast<uint16_t>(m[r] >> (16 * lane));
          }
          if (lane < 16) {
            uint32_t v = 0;
#pragma unroll
            for (int qd = 0; qd < 4; ++qd)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                v |= static_cast<uint32_t>((m[r] >> (16 * qd + lane)) & 1ull) << (4 * qd + r);
            tbits[64 * wn + 16 * j + lane][4 * wm + i] = static_cast<uint16_t>(v);
          }
        }
      }
    }
    __syncthreads();
    write_tile_words(c, dbits, tbits, bitmask, bm_off[c.e]);
    __syncthreads();
  }
}

// float32 tokens: same tiles and bitmask, plain FMA with an 8x8 micro-tile
// per thread.
__global__ __launch_bounds__(256) void gram_kernel_f32(
    const float* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, float h,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask) {
  constexpr int KC = 16;
  __shared__ float Ps[kTile][KC + 1];
  __shared__ float Qs[kTile][KC + 1];
  __shared__ uint8_t edge[kTile][kTile];
  __shared__ uint16_t dbits[kTile][8];
  __shared__ uint16_t tbits[kTile][8];
  __shared__ float inv_a[kTile], inv_b[kTile];
  if (*err) return;
  const int tid = threadIdx.x;
  const int rb = (tid >> 4) * 8, cb = (tid & 15) * 8;
  const int total = tile_off[E];
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const TileCoord c = decode_tile(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    if (tid < kTile) inv_a[tid] = inv_norm[pt[min(c.ti * kTile + tid, c.n - 1)]];
    else inv_b[tid - kTile] = inv_norm[pt[min(c.tj * kTile + tid - kTile, c.n - 1)]];
    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
    for (int k0 = 0; k0 < d; k0 += KC) {
      __syncthreads();
      for (int idx = tid; idx < kTile * KC; idx += 256) {
        const int r = idx / KC, kk = idx % KC;
        const int a = min(c.ti * kTile + r, c.n - 1);
        const int b = min(c.tj * kTile + r, c.n - 1);
        Ps[r][kk] = X[static_cast<size_t>(pt[a]) * d + k0 + kk];
        Qs[r][kk] = X[static_cast<size_t>(pt[b]) * d + k0 + kk];
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < KC; ++kk) {
        float pa[8], qb[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) pa[i] = Ps[rb + i][kk];
#pragma unroll
        for (int j = 0; j < 8; ++j) qb[j] = Qs[cb + j][kk];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(pa[i], qb[j], acc[i][j]);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int a = c.ti * kTile + rb + i, b = c.tj * kTile + cb + j;
        const float cs = acc[i][j] * inv_a[rb + i] * inv_b[cb + j];
        edge[rb + i][cb + j] = (a < c.n && b < c.n && a != b && cs >= h) ? 1 : 0;
      }
    __syncthreads();
    for (int idx = tid; idx < kTile * 8; idx += 256) {
      const int r = idx >> 3, g = idx & 7;
      uint32_t dv = 0, tv = 0;
      for (int bit = 0; bit < 16; ++bit) {
        dv |= static_cast<uint32_t>(edge[r][16 * g + bit]) << bit;
        tv |= static_cast<uint32_t>(edge[16 * g + bit][r]) << bit;
      }
      dbits[r][g] = static_cast<uint16_t>(dv);
      tbits[r][g] = static_cast<uint16_t>(tv);
    }
    __syncthreads();
    write_tile_words(c, dbits, tbits, bitmask, bm_off[c.e]);
  }
}

__global__ __launch_bounds__(256) void degree_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg,
    int32_t* __restrict__ state, int32_t* __restrict__ degree_out) {
  if (*err) return;
  const int lane = threadIdx.x & 63;
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= offsets[E]) return;
  const int e = bucket_of(offsets, E, p);
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  const uint64_t* row = bitmask + bm_off[e] + static_cast<long long>(p - lo) * W;
  int cnt = 0;
  for (int wd = lane; wd < W; wd += 64) cnt += __popcll(row[wd]);
  cnt = wave_sum_i32(cnt);
  if (lane == 0) {
    deg[p] = cnt;
    state[p] = kStateUndecided;
    if (degree_out) degree_out[p] = cnt;
  }
}

// Decides position p if its neighbours allow it; returns true when p is
// still undecided afterwards (wave-uniform).
__device__ __forceinline__ bool greedy_visit(int p, int lo, int n, int W,
                                             const uint64_t* __restrict__ row,
                                             const int32_t* __restrict__ deg, int32_t* state) {
  const int lane = threadIdx.x & 63;
  const int dp = deg[p];
  bool kept_nb = false, blocked = false;
  for (int wd = lane; wd < W && !kept_nb; wd += 64) {
    uint64_t bits = row[wd];
    while (bits) {
      const int b = __ffsll(static_cast<long long>(bits)) - 1;
      bits &= bits - 1;
      if (wd * 64 + b >= n) break;   // defensive: no bit lies past the bucket
      const int q = lo + wd * 64 + b;
      const int st = load_flag(&state[q]);
      if (st == kStateKept) { kept_nb = true; break; }
      if (st == kStateUndecided) {
        const int dq = deg[q];
        if (dq > dp || (dq == dp && q < p)) blocked = true;
      }
    }
  }
  const bool any_kept = __ballot(kept_nb) != 0;
  const bool any_blocked = __ballot(blocked) != 0;
  if (any_kept) {
    if (lane == 0) store_flag(&state[p], kStateAbsorbed);
    return false;
  }
  if (!any_blocked) {
    if (lane == 0) store_flag(&state[p], kStateKept);
    return false;
  }
  return true;
}

__global__ __launch_bounds__(256) void greedy_round_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state) {
  if (*err) return;
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= offsets[E]) return;
  if (load_flag(&state[p]) != kStateUndecided) return;
  const int e = bucket_of(offsets, E, p);
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  greedy_visit(p, lo, n, W, bitmask + bm_off[e] + static_cast<long long>(p - lo) * W, deg, state);
}

// One workgroup per bucket: rounds until every position is decided.  Each
// round decides at least the highest-priority undecided position, so at most
// n rounds run.
__global__ __launch_bounds__(1024) void greedy_finish_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state) {
  if (*err) return;
  const int e = blockIdx.x;
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  if (n == 0) return;
  const int wv = threadIdx.x >> 6;
  for (int it = 0; it <= n; ++it) {
    int undecided = 0;
    for (int pl = wv; pl < n; pl += 16) {
      const int p = lo + pl;
      if (load_flag(&state[p]) != kStateUndecided) continue;
      if (greedy_visit(p, lo, n, W, bitmask + bm_off[e] + static_cast<long long>(pl) * W, deg, state))
        undecided = 1;
    }
    if (!__syncthreads_or(undecided)) break;
  }
}

__global__ __launch_bounds__(256) void assign_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, const int32_t* __restrict__ state,
    int32_t* __restrict__ rep_of_pos) {
  const int lane = threadIdx.x & 63;
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (p >= offsets[E]) return;
  // after a layout error nothing was decided: every position keeps itself
  if (*err || state[p] != kStateAbsorbed) {
    if (lane == 0) rep_of_pos[p] = p;
    return;
  }
  const int e = bucket_of(offsets, E, p);
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  const uint64_t* row = bitmask + bm_off[e] + static_cast<long long>(p - lo) * W;
  // priority key: higher degree first, then lower position
  unsigned long long best = 0;
  for (int wd = lane; wd < W; wd += 64) {
    uint64_t bits = row[wd];
    while (bits) {
      const int b = __ffsll(static_cast<long long>(bits)) - 1;
      bits &= bits - 1;
      if (wd * 64 + b >= n) break;
      const int q = lo + wd * 64 + b;
      if (state[q] == kStateKept) {
        const unsigned long long key = (static_cast<unsigned long long>(deg[q]) << 32) |
                                       static_cast<unsigned int>(~static_cast<unsigned int>(q));
        best = key > best ? key : best;
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned long long other = __shfl_xor(best, o, 64);
    best = other > best ? other : best;
  }
  if (lane == 0) rep_of_pos[p] = static_cast<int>(~static_cast<unsigned int>(best & 0xffffffffull));
}

// One workgroup: rep_index[p] = number of representatives before p,
// rep_token[row] = token of that representative, rep_offsets per expert.
__global__ __launch_bounds__(1024) void rep_scan_kernel(
    const int32_t* __restrict__ offsets, int E, const int32_t* __restrict__ rep_of_pos,
    const int32_t* __restrict__ perm_token, int32_t* rep_index, int32_t* __restrict__ rep_token,
    int32_t* __restrict__ rep_offsets) {
  constexpr int ITEMS = 16;
  __shared__ int wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int S = offsets[E];
  int carry = 0;
  for (int base = 0; base < S; base += 1024 * ITEMS) {
    int f[ITEMS];
    int local = 0;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int p = base + tid * ITEMS + i;
      f[i] = (p < S && rep_of_pos[p] == p) ? 1 : 0;
      local += f[i];
    }
    int incl = local;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int wbase = 0, chunk_total = 0;
    for (int i = 0; i < 16; ++i) {
      const int v = wsum[i];
      if (i < wv) wbase += v;
      chunk_total += v;
    }
    int r = carry + wbase + incl - local;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int p = base + tid * ITEMS + i;
      if (p < S) {
        rep_index[p] = r;
        if (f[i]) rep_token[r] = perm_token[p];
        r += f[i];
      }
    }
    carry += chunk_total;
    __syncthreads();
  }
  __threadfence();
  __syncthreads();
  if (tid <= E) {
    const int p = offsets[tid];
    rep_offsets[tid] = (p < S) ? load_flag(&rep_index[p]) : carry;
  }
}

__global__ __launch_bounds__(256) void rep_row_kernel(const int32_t* __restrict__ offsets, int E,
                                                      const int32_t* __restrict__ rep_of_pos,
                                                      const int32_t* __restrict__ rep_index,
                                                      int32_t* __restrict__ rep_row) {
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (p >= offsets[E]) return;
  rep_row[p] = rep_index[rep_of_pos[p]];
}

__global__ __launch_bounds__(256) void gather_kernel(const uint8_t* __restrict__ x, size_t row_bytes,
                                                     const int32_t* __restrict__ rep_offsets, int E,
                                                     const int32_t* __restrict__ rep_token,
                                                     uint8_t* __restrict__ x_rep) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rep_offsets[E]) return;
  const uint4* src = reinterpret_cast<const uint4*>(x + static_cast<size_t>(rep_token[r]) * row_bytes);
  uint4* dst = reinterpret_cast<uint4*>(x_rep + static_cast<size_t>(r) * row_bytes);
  for (size_t i = lane; i < row_bytes / 16; i += 64) dst[i] = src[i];
}

struct CondenseWs {
  float* inv_norm;
  int32_t* tile_off;
  long long* bm_off;
  int* err;
  int32_t* deg;
  int32_t* state;
  int32_t* rep_index;
  uint64_t* bitmask;
  long long cap_words;
};

CondenseWs carve_condense(Carver& c, int T, int E, int k, int max_bucket) {
  CondenseWs w;
  const long long S = static_cast<long long>(T) * k;
  w.inv_norm = c.take<float>(T);
  w.tile_off = c.take<int32_t>(E + 1);
  w.bm_off = c.take<long long>(E + 1);
  w.err = c.take<int>(1);
  w.deg = c.take<int32_t>(S);
  w.state = c.take<int32_t>(S);
  w.rep_index = c.take<int32_t>(S);
  w.cap_words = S * ((static_cast<long long>(max_bucket) + 63) / 64);
  w.bitmask = c.take<uint64_t>(static_cast<size_t>(w.cap_words));
  return w;
}

int gram_grid() {
  static int grid = 0;
  if (!grid) {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    grid = 2 * cus;
  }
  return grid;
}

}  // namespace
}  // namespace luffy

using namespace luffy;

extern "C" size_t luffy_condense_workspace_size(int T, int d, int E, int k, int max_bucket) {
  (void)d;
  if (T <= 0 || E <= 0 || k <= 0 || max_bucket < 0) return 0;
  Carver c(nullptr);
  carve_condense(c, T, E, k, max_bucket);
  return c.size();
}

extern "C" int luffy_condense(const void* x, int T, int d, int dtype,
                              const int32_t* perm_token, const int32_t* offsets,
                              int E, int k, int max_bucket, float threshold,
                              int32_t* rep_of_pos, int32_t* rep_row,
                              int32_t* rep_offsets, int32_t* rep_token,
                              void* x_rep, int32_t* degree,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !perm_token || !offsets || !rep_of_pos || !rep_row || !rep_offsets || !rep_token)
    return fail(LUFFY_E_INVALID, "luffy_condense: null pointer argument");
  if (T <= 0 || d <= 0 || E <= 0 || max_bucket < 0)
    return fail(LUFFY_E_INVALID, "luffy_condense: T=%d d=%d E=%d max_bucket=%d", T, d, E, max_bucket);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "luffy_condense: k=%d must be 1 or 2", k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_condense: unknown dtype %d", dtype);
  if (threshold != threshold) return fail(LUFFY_E_INVALID, "luffy_condense: threshold is NaN");
  if (E > kMaxExperts) return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: E=%d > %d", E, kMaxExperts);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: d=%d not a multiple of 64", d);
  if (static_cast<long long>(T) * k >= (1ll << 31))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: T*k too large");
  const size_t need = luffy_condense_workspace_size(T, d, E, k, max_bucket);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_condense: workspace needs %zu bytes, 256-aligned", need);

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  CondenseWs ws = carve_condense(c, T, E, k, max_bucket);
  const int S = T * k;
  const bool bf16 = dtype == LUFFY_BF16;

  {
    ProfileScope prof_("norm", s);
    if (bf16) norm_kernel<true><<<(T + 3) / 4, 256, 0, s>>>(x, T, d, ws.inv_norm);
    else norm_kernel<false><<<(T + 3) / 4, 256, 0, s>>>(x, T, d, ws.inv_norm);
  }
  {
    ProfileScope prof_("gram_prep", s);
    gram_prep_kernel<<<1, 64, 0, s>>>(offsets, E, max_bucket, ws.cap_words, ws.tile_off, ws.bm_off, ws.err);
  }
  {
    ProfileScope prof_("gram", s);
    if (bf16)
      gram_kernel_bf16<<<gram_grid(), 256, 0, s>>>(static_cast<const uint16_t*>(x), d, perm_token, offsets, E,
                                                 ws.inv_norm, threshold, ws.tile_off, ws.bm_off, ws.err,
                                                 ws.bitmask);
    else
      gram_kernel_f32<<<gram_grid(), 256, 0, s>>>(static_cast<const float*>(x), d, perm_token, offsets, E,
                                                  ws.inv_norm, threshold, ws.tile_off, ws.bm_off, ws.err,
                                                  ws.bitmask);
  }
  const int wave_blocks = (S + 3) / 4;
  {
    ProfileScope prof_("degree", s);
    degree_kernel<<<wave_blocks, 256, 0, s>>>(offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.state, degree);
  }
  for (int r = 0; r < kGreedyGridRounds; ++r) {
    ProfileScope prof_("greedy_round", s);
    greedy_round_kernel<<<wave_blocks, 256, 0, s>>>(offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.state);
  }
  {
    ProfileScope prof_("greedy_finish", s);
    greedy_finish_kernel<<<E, 1024, 0, s>>>(offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.state);
  }
  {
    ProfileScope prof_("assign", s);
    assign_kernel<<<wave_blocks, 256, 0, s>>>(offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.state, rep_of_pos);
  }
  {
    ProfileScope prof_("rep_scan", s);
    rep_scan_kernel<<<1, 1024, 0, s>>>(offsets, E, rep_of_pos, perm_token, ws.rep_index, rep_token, rep_offsets);
  }
  {
    ProfileScope prof_("rep_row", s);
    rep_row_kernel<<<(S + 255) / 256, 256, 0, s>>>(offsets, E, rep_of_pos, ws.rep_index, rep_row);
  }
  if (x_rep) {
    ProfileScope prof_("gather", s);
    gather_kernel<<<wave_blocks, 256, 0, s>>>(static_cast<const uint8_t*>(x),
                                              static_cast<size_t>(d) * elem_bytes(dtype), rep_offsets, E,
                                              rep_token, static_cast<uint8_t*>(x_rep));
  }
  return check_launch("luffy_condense");
}
