// luffy_condense: per-bucket cosine threshold graph, representative
// selection and compaction.
//
// Kernels, in launch order:
//   norm_kernel          1/|x_t| per token (one wave per row); clears the
//                        degree counters and walk states; its first wave
//                        lays out every bucket's tiles and bitmask.
//   gram_kernel_{bf16,f32}  persistent loop over the upper-triangle tiles
//                        (256 rows bf16, 128 rows fp32) of every bucket's Gram
//                        matrix.  The epilogue turns cos >= h into adjacency
//                        bits, writes both the tile and its transpose (every
//                        bitmask word is written exactly once) and adds each
//                        row's edge count to its degree.
//   greedy_round_kernel  one round of the parallel form of the greedy walk,
//                        16 lanes per position (launched twice, which
//                        decides every position of a union of cliques;
//                        decided positions return at once).
//   greedy_finish_kernel one workgroup per bucket repeats rounds until the
//                        bucket is fully decided (after a coalesced check
//                        that anything is left).
//   claim_kernel         every kept position offers itself to its
//                        neighbours (64-bit atomic max of degree, ~position):
//                        an absorbed position ends with its first-visited
//                        kept neighbour.
//   rep_local_kernel, rep_finalize_kernel  representative rows by a two-pass
//                        scan: rep_row, rep_token, rep_offsets.
//   gather_kernel        optional copy of the representative rows.
//
// The walk of Sec. 5.2 visits positions by priority (degree descending,
// position ascending) and keeps a position iff no neighbour of higher
// priority was kept.  In parallel: an undecided position whose kept
// neighbour exists is absorbed; one whose every higher-priority neighbour is
// absorbed is kept.  Both rules only read final decisions, so rounds may see
// each other's updates early without changing the result, and every round
// decides at least the highest-priority undecided position.
#include <algorithm>

#include "gemm_core.h"
#include "luffy_common.h"

namespace luffy {
namespace {

constexpr int kGreedyGridRounds = 2;
constexpr int kTile = 256;      // similarity tile of the bf16 path (GramGemm)
constexpr int kTileF32 = 64;    // similarity tile of the fp32 path
constexpr int kGroupsF32 = kTileF32 / 16;   // 16-column bit groups per tile row
constexpr int kWordsF32 = kTileF32 / 64;    // bitmask words per tile row
constexpr int kStateUndecided = 0, kStateKept = 1, kStateAbsorbed = 2;

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

// Tile and bitmask layout of every bucket, by one wave (lane e: expert e,
// E <= 64).  Flags an error (and schedules no tile) when a bucket exceeds
// max_bucket or the bitmask exceeds the workspace.
__device__ __forceinline__ void gram_layout(const int32_t* __restrict__ offsets, int E, int max_bucket,
                                            int tile, long long cap_words, int32_t* __restrict__ tile_off,
                                            long long* __restrict__ bm_off, int* __restrict__ err) {
  const int lane = threadIdx.x & 63;
  const int n = lane < E ? offsets[lane + 1] - offsets[lane] : 0;
  const int nt = (n + tile - 1) / tile;
  const int tiles = nt * (nt + 1) / 2;
  const long long words = static_cast<long long>(n) * ((n + 63) / 64);
  int tincl = tiles;
  long long wincl = words;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int tu = __shfl_up(tincl, o, 64);
    const long long wu = __shfl_up(wincl, o, 64);
    if (lane >= o) {
      tincl += tu;
      wincl += wu;
    }
  }
  const long long wtotal = __shfl(wincl, 63, 64);
  const bool bad = __ballot(lane < E && (n < 0 || n > max_bucket)) != 0 || wtotal > cap_words;
  if (lane < E) {
    tile_off[lane] = bad ? 0 : tincl - tiles;
    bm_off[lane] = wincl - words;
  }
  if (lane == 63) {
    tile_off[E] = bad ? 0 : tincl;
    bm_off[E] = wincl;
    *err = bad ? 1 : 0;
  }
}

// NORMS = false: the norms were computed by the caller (luffy_route); only
// the clearing and the layout run.
template <bool BF16, bool NORMS>
__global__ __launch_bounds__(256) void norm_kernel(const void* __restrict__ xv, int T, int d,
                                                   float* __restrict__ inv_norm, int S,
                                                   int32_t* __restrict__ deg, int32_t* __restrict__ state,
                                                   unsigned long long* __restrict__ claim,
                                                   const int32_t* __restrict__ offsets, int E, int max_bucket,
                                                   int tile, long long cap_words, int32_t* __restrict__ tile_off,
                                                   long long* __restrict__ bm_off, int* __restrict__ err) {
  if (blockIdx.x == 0 && threadIdx.x < 64)
    gram_layout(offsets, E, max_bucket, tile, cap_words, tile_off, bm_off, err);
  // also clears the degree counters, walk states and claim keys of all S positions
  for (int p = blockIdx.x * 256 + threadIdx.x; p < S; p += gridDim.x * 256) {
    deg[p] = 0;
    state[p] = 0;
    claim[p] = 0ull;
  }
  if constexpr (!NORMS) return;
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

struct TileCoord {
  int e, ti, tj, lo, n, W;
};

// Bucket of tile `tile` (the last e with tile_off[e] <= tile, skipping
// empty buckets), its first tile, first slot and size.  One load per lane
// (lane e holds bucket e, E <= 64) and a ballot: a single round trip instead
// of a walk of dependent loads.  Called by whole waves.
__device__ __forceinline__ void locate_bucket(int tile, const int32_t* __restrict__ tile_off,
                                              const int32_t* __restrict__ offsets, int E, int& e, int& tbase,
                                              int& lo, int& n) {
  const int lane = threadIdx.x & 63;
  const bool in = lane < E;
  const int to = in ? tile_off[lane] : 0;
  const int o0 = in ? offsets[lane] : 0;
  const int o1 = in ? offsets[lane + 1] : 0;
  e = __popcll(__ballot(in && lane >= 1 && to <= tile));
  tbase = __builtin_amdgcn_readfirstlane(__shfl(to, e, 64));
  lo = __builtin_amdgcn_readfirstlane(__shfl(o0, e, 64));
  n = __builtin_amdgcn_readfirstlane(__shfl(o1, e, 64)) - lo;
}

__device__ __forceinline__ TileCoord decode_tile(int tile, const int32_t* __restrict__ tile_off,
                                                 const int32_t* __restrict__ offsets, int E) {
  TileCoord c;
  int tbase;
  locate_bucket(tile, tile_off, offsets, E, c.e, tbase, c.lo, c.n);
  const int q = tile - tbase;
  int tj = static_cast<int>((sqrtf(8.0f * q + 1.0f) - 1.0f) * 0.5f);
  while (tj * (tj + 1) / 2 > q) --tj;
  while ((tj + 1) * (tj + 2) / 2 <= q) ++tj;
  c.tj = tj;
  c.ti = q - tj * (tj + 1) / 2;
  c.W = (c.n + 63) / 64;
  return c;
}

// Writes the tile's adjacency words: rows of tile-row ti at words
// kWordsF32 * tj + w (from dbits) and, off the diagonal, rows of tile-row tj
// at words kWordsF32 * ti + w (from tbits).  dbits/tbits: [kTileF32 rows]
// [kGroupsF32 groups of 16 columns].
__device__ __forceinline__ void write_tile_words(const TileCoord& c, const uint16_t (*dbits)[kGroupsF32],
                                                 const uint16_t (*tbits)[kGroupsF32],
                                                 uint64_t* __restrict__ bitmask, long long base) {
  const int tid = threadIdx.x;
  if (tid >= kTileF32 * kWordsF32) return;
  const int rl = tid / kWordsF32, ww = tid % kWordsF32;
  auto pack = [](const uint16_t* g) {
    return static_cast<uint64_t>(g[0]) | (static_cast<uint64_t>(g[1]) << 16) |
           (static_cast<uint64_t>(g[2]) << 32) | (static_cast<uint64_t>(g[3]) << 48);
  };
  {
    const int a = c.ti * kTileF32 + rl;
    const int wd = kWordsF32 * c.tj + ww;
    if (a < c.n && wd < c.W)
      bitmask[base + static_cast<long long>(a) * c.W + wd] = pack(&dbits[rl][4 * ww]);
  }
  if (c.ti != c.tj) {
    const int b = c.tj * kTileF32 + rl;
    const int wd = kWordsF32 * c.ti + ww;
    if (b < c.n && wd < c.W)
      bitmask[base + static_cast<long long>(b) * c.W + wd] = pack(&tbits[rl][4 * ww]);
  }
}

// Tile order inside a bucket for the 256-row tiles: columns are taken in
// groups of 4; inside a group the tiles go row by row (ti major), first the
// full rows above the group's diagonal block, then its upper triangle.  Any
// 32 consecutive tiles then cover about 8 row blocks x 4 column blocks, so
// the blocks of one XCD that run them together share operand rows in L2.
__device__ __forceinline__ TileCoord decode_tile_grouped(int tile, const int32_t* __restrict__ tile_off,
                                                         const int32_t* __restrict__ offsets, int E) {
  TileCoord c;
  int tbase;
  locate_bucket(tile, tile_off, offsets, E, c.e, tbase, c.lo, c.n);
  c.W = (c.n + 63) / 64;
  const int nt = (c.n + kTile - 1) / kTile;
  const int q = tile - tbase;
  // tiles before column group g: 8g^2 + 2g
  int g = static_cast<int>((sqrtf(4.0f + 32.0f * q) - 2.0f) / 16.0f);
  while (g > 0 && 8 * g * g + 2 * g > q) --g;
  while (8 * (g + 1) * (g + 1) + 2 * (g + 1) <= q) ++g;
  const int r = q - (8 * g * g + 2 * g);
  const int wdt = min(4, nt - 4 * g);
  if (r < 4 * g * wdt) {
    c.ti = r / wdt;
    c.tj = 4 * g + r % wdt;
  } else {
    int r2 = r - 4 * g * wdt, i = 0;
    while (r2 >= wdt - i) { r2 -= wdt - i; ++i; }
    c.ti = 4 * g + i;
    c.tj = 4 * g + i + r2;
  }
  return c;
}

// v_writelane_b32: `old` with lane `lane` replaced by the wave-uniform
// `value` (the LLVM intrinsic, which clang does not expose as a builtin).
__device__ int amdgcn_writelane(int value, int lane, int old) __asm("llvm.amdgcn.writelane");

using GramGemm = GemmBig64;
static_assert(GramGemm::BM == kTile && GramGemm::BN == kTile, "similarity tile");

__global__ __launch_bounds__(GramGemm::THREADS) void gram_kernel_bf16(
    const uint16_t* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, float h,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg) {
  using G = GramGemm;
  __shared__ __attribute__((aligned(16))) uint8_t lds[G::LDS_BYTES];
  __shared__ __attribute__((aligned(16))) float inv_a[kTile];
  __shared__ float inv_b[kTile];
  // after the K loop the operand buffers hold the tile's adjacency pieces:
  // dbits[row][32-column group], tbits[column][32-row group]
  uint32_t (*dbits)[kTile / 32] = reinterpret_cast<uint32_t (*)[kTile / 32]>(lds);
  uint32_t (*tbits)[kTile / 32] = reinterpret_cast<uint32_t (*)[kTile / 32]>(lds + kTile * kTile / 8);
  if (*err) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = G::wave_m(w), wn = G::wave_n(w);
  const int total = tile_off[E];
  for (int tile = xcd_virtual_block(); tile < total; tile += gridDim.x) {
    const TileCoord c = decode_tile_grouped(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    uint32_t poff[G::LP], qoff[G::LQ];
#pragma unroll
    for (int j = 0; j < G::LP; ++j)
      poff[j] = static_cast<uint32_t>(pt[min(c.ti * kTile + G::load_row(j), c.n - 1)]) * d;
#pragma unroll
    for (int j = 0; j < G::LQ; ++j)
      qoff[j] = static_cast<uint32_t>(pt[min(c.tj * kTile + G::load_row(G::LP + j) - G::BM, c.n - 1)]) * d;
    for (int i = tid; i < 2 * kTile; i += G::THREADS) {
      if (i < kTile) inv_a[i] = inv_norm[pt[min(c.ti * kTile + i, c.n - 1)]];
      else inv_b[i - kTile] = inv_norm[pt[min(c.tj * kTile + i - kTile, c.n - 1)]];
    }
    G::Acc acc;
    G::zero(acc);
    G::run(X, poff, X, qoff, d, c.n - c.ti * kTile, c.n - c.tj * kTile, lds, acc);  // ends with a barrier

    // Each (fm, fn) block is 32 x 32.  Lane l holds column bbase + l%32 and,
    // in accumulator v, row abase + rv(v) + 4*(l/32), rv(v) = 8(v/4) + v%4.
    // Ballot v is then two row pieces: bits 0..31 are the columns of row
    // abase + rv(v), bits 32..63 those of row abase + rv(v) + 4; lane r < 32
    // receives row r's piece by writelane.  The column piece of column
    // bbase + c has bit rv(v) (+4 in the upper half-wave) from accumulator v:
    // each lane assembles its 16 bits with selects on its own compares, and
    // lanes c and c+32 merge theirs with one cross-half exchange.  Every piece
    // of the tile is written exactly once.  Edge test:
    // dot * (1/|a|) * (1/|b|) >= h, for rows and columns inside the bucket,
    // never a token with itself.
    const int l31 = lane & 31, hi = lane >> 5;
    const bool same_tile = c.ti == c.tj;
    const int nrow_a = c.n - c.ti * kTile, nrow_b = c.n - c.tj * kTile;
#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm) {
      const int abase = wm * G::WTM + 32 * fm;
      // this lane's 16 rows: abase + 8q + 4hi + r, as 4 runs of 4.  Rows
      // (and columns) outside the bucket get a NaN scale, which fails every
      // comparison.
      const float nan = __builtin_nanf("");
      float ia[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int al0 = abase + 8 * q + 4 * hi;
        const float4 f = *reinterpret_cast<const float4*>(&inv_a[al0]);
        const float fv[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) ia[4 * q + r] = al0 + r < nrow_a ? fv[r] : nan;
      }
#pragma unroll
      for (int fn = 0; fn < G::FN; ++fn) {
        const int bbase = wn * G::WTN + 32 * fn;
        const int bl = bbase + l31;
        const float ib = bl < nrow_b ? inv_b[bl] : nan;
        const bool diag = same_tile && abase == bbase;   // wave-uniform
        uint32_t colbits = 0, piece = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int rv = 8 * (v >> 2) + (v & 3);
          bool e = acc[fm][fn][v] * ia[v] * ib >= h;
          if (diag) e = e && rv + 4 * hi != l31;
          const uint64_t m = __ballot(e);
          piece = amdgcn_writelane(static_cast<int>(static_cast<uint32_t>(m)), rv, piece);
          piece = amdgcn_writelane(static_cast<int>(static_cast<uint32_t>(m >> 32)), rv + 4, piece);
          colbits |= e ? 1u << rv : 0u;
        }
        colbits <<= 4 * hi;
        const uint32_t tv = colbits | static_cast<uint32_t>(__shfl_xor(static_cast<int>(colbits), 32, 64));
        if (lane < 32) {
          dbits[abase + l31][bbase >> 5] = piece;
          tbits[bl][abase >> 5] = tv;
        }
      }
    }
    __syncthreads();
    // degree: edges of each tile row (and, off the diagonal, of each mirrored row)
    for (int i = tid; i < 2 * kTile; i += G::THREADS) {
      const bool mirror = i >= kTile;
      const int rl = mirror ? i - kTile : i;
      const uint32_t* pcs = mirror ? tbits[rl] : dbits[rl];
      int cnt = 0;
#pragma unroll
      for (int g = 0; g < kTile / 32; ++g) cnt += __popc(pcs[g]);
      const int r = (mirror ? c.tj : c.ti) * kTile + rl;
      if (cnt && r < c.n && (!mirror || c.ti != c.tj)) atomicAdd(&deg[c.lo + r], cnt);
    }
    // write the words: 4 per row of the tile, direct and (off-diagonal) mirrored
    for (int i = tid; i < kTile * 4; i += G::THREADS) {
      const int rl = i >> 2, ww = i & 3;
      const uint64_t dv = static_cast<uint64_t>(dbits[rl][2 * ww]) |
                          (static_cast<uint64_t>(dbits[rl][2 * ww + 1]) << 32);
      const int a = c.ti * kTile + rl, wd = 4 * c.tj + ww;
      if (a < c.n && wd < c.W) bitmask[bm_off[c.e] + static_cast<long long>(a) * c.W + wd] = dv;
      if (c.ti != c.tj) {
        const uint64_t tv = static_cast<uint64_t>(tbits[rl][2 * ww]) |
                            (static_cast<uint64_t>(tbits[rl][2 * ww + 1]) << 32);
        const int bb = c.tj * kTile + rl, wt = 4 * c.ti + ww;
        if (bb < c.n && wt < c.W) bitmask[bm_off[c.e] + static_cast<long long>(bb) * c.W + wt] = tv;
      }
    }
    __syncthreads();
  }
}

// float32 tokens: 64-row tiles (small buckets give more tiles than with the
// bf16 path's 256), same bitmask, plain FMA with a 4x4 micro-tile per
// thread.
__global__ __launch_bounds__(256) void gram_kernel_f32(
    const float* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, float h,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg) {
  constexpr int KC = 16;
  __shared__ float Ps[kTileF32][KC + 1];
  __shared__ float Qs[kTileF32][KC + 1];
  constexpr int MT = kTileF32 / 16;   // micro-tile edge: 16 x 16 threads cover the tile
  __shared__ uint8_t edge[kTileF32][kTileF32];
  __shared__ uint16_t dbits[kTileF32][kGroupsF32];
  __shared__ uint16_t tbits[kTileF32][kGroupsF32];
  __shared__ float inv_a[kTileF32], inv_b[kTileF32];
  if (*err) return;
  const int tid = threadIdx.x;
  const int rb = (tid >> 4) * MT, cb = (tid & 15) * MT;
  const int total = tile_off[E];
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const TileCoord c = decode_tile(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    if (tid < kTileF32) inv_a[tid] = inv_norm[pt[min(c.ti * kTileF32 + tid, c.n - 1)]];
    else if (tid < 2 * kTileF32) inv_b[tid - kTileF32] = inv_norm[pt[min(c.tj * kTileF32 + tid - kTileF32, c.n - 1)]];
    // staged element i of this thread: tile row r0 + 16i, column kk; the
    // token rows are looked up once per tile and the next chunk is loaded
    // into registers while the current one is multiplied
    constexpr int PER = kTileF32 * KC / 256;
    const int kk = tid % KC, r0 = tid / KC;
    const float* pp[PER];
    const float* qp[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int r = r0 + (256 / KC) * i;
      pp[i] = X + static_cast<size_t>(pt[min(c.ti * kTileF32 + r, c.n - 1)]) * d + kk;
      qp[i] = X + static_cast<size_t>(pt[min(c.tj * kTileF32 + r, c.n - 1)]) * d + kk;
    }
    float vp[PER], vq[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      vp[i] = pp[i][0];
      vq[i] = qp[i][0];
    }
    float acc[MT][MT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < MT; ++j) acc[i][j] = 0.f;
    for (int k0 = 0; k0 < d; k0 += KC) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        Ps[r0 + (256 / KC) * i][kk] = vp[i];
        Qs[r0 + (256 / KC) * i][kk] = vq[i];
      }
      __syncthreads();
      if (k0 + KC < d) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
          vp[i] = pp[i][k0 + KC];
          vq[i] = qp[i][k0 + KC];
        }
      }
#pragma unroll
      for (int k = 0; k < KC; ++k) {
        float pa[MT], qb[MT];
#pragma unroll
        for (int i = 0; i < MT; ++i) pa[i] = Ps[rb + i][k];
#pragma unroll
        for (int j = 0; j < MT; ++j) qb[j] = Qs[cb + j][k];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < MT; ++j) acc[i][j] = fmaf(pa[i], qb[j], acc[i][j]);
      }
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        const int a = c.ti * kTileF32 + rb + i, b = c.tj * kTileF32 + cb + j;
        const float cs = acc[i][j] * inv_a[rb + i] * inv_b[cb + j];
        edge[rb + i][cb + j] = (a < c.n && b < c.n && a != b && cs >= h) ? 1 : 0;
      }
    __syncthreads();
    for (int idx = tid; idx < kTileF32 * kGroupsF32; idx += 256) {
      const int r = idx / kGroupsF32, g = idx % kGroupsF32;
      uint32_t dv = 0, tv = 0;
      for (int bit = 0; bit < 16; ++bit) {
        dv |= static_cast<uint32_t>(edge[r][16 * g + bit]) << bit;
        tv |= static_cast<uint32_t>(edge[16 * g + bit][r]) << bit;
      }
      dbits[r][g] = static_cast<uint16_t>(dv);
      tbits[r][g] = static_cast<uint16_t>(tv);
    }
    __syncthreads();
    if (tid < 2 * kTileF32) {
      const bool mirror = tid >= kTileF32;
      const int rl = mirror ? tid - kTileF32 : tid;
      int cnt = 0;
      for (int g = 0; g < kGroupsF32; ++g) cnt += __popc(mirror ? tbits[rl][g] : dbits[rl][g]);
      const int r = (mirror ? c.tj : c.ti) * kTileF32 + rl;
      if (cnt && r < c.n && (!mirror || c.ti != c.tj)) atomicAdd(&deg[c.lo + r], cnt);
    }
    write_tile_words(c, dbits, tbits, bitmask, bm_off[c.e]);
  }
}

// Decides position p if its neighbours allow it; returns true when p is
// still undecided afterwards (uniform over the GW-lane group that visits p,
// GW = 16 or 64, aligned inside the wave).  The group walks the adjacency
// row 4*GW words at a time (four word loads in flight per lane), gathers the
// state and degree of up to 8 neighbours at a time before testing them, and
// stops after the first batch of words that shows a kept neighbour (p is
// absorbed) or an undecided neighbour of higher priority (p stays
// undecided for a later round).  The grid
// rounds use plain loads (FRESH = false): a state written by another XCD in
// the same launch may be seen late, which only delays a decision (states
// change once, from undecided to final).  The single-workgroup finishing
// pass, which relies on seeing the previous iteration's decisions, reads
// the states with coherent atomic loads (FRESH = true).
template <bool FRESH, int GW>
__device__ __forceinline__ bool greedy_visit(int p, int lo, int n, int W,
                                             const uint64_t* __restrict__ row,
                                             const int32_t* __restrict__ deg, int32_t* state) {
  const int lane = threadIdx.x & 63;
  const int gl = lane & (GW - 1);
  const int gshift = lane & ~(GW - 1);
  const uint64_t gmask = GW == 64 ? ~0ull : ((1ull << (GW & 63)) - 1);
  const int dp = deg[p];
  bool kept_nb = false, blocked = false;
  for (int b0 = 0; b0 < W; b0 += 4 * GW) {
    const int wd0 = b0 + gl;
    uint64_t wv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) wv[u] = wd0 + GW * u < W ? row[wd0 + GW * u] : 0ull;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint64_t bits = wv[u];
      const int cbase = (wd0 + GW * u) * 64;
      while (bits) {
        int q[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          q[i] = -1;
          if (bits) {
            const int b = __ffsll(static_cast<long long>(bits)) - 1;
            bits &= bits - 1;
            if (cbase + b < n) q[i] = lo + cbase + b;   // no bit lies past the bucket
          }
        }
        int st[8], dq[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          st[i] = q[i] >= 0 ? (FRESH ? load_flag(&state[q[i]]) : state[q[i]]) : kStateAbsorbed;
          dq[i] = q[i] >= 0 ? deg[q[i]] : 0;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (st[i] == kStateKept) kept_nb = true;
          else if (st[i] == kStateUndecided && (dq[i] > dp || (dq[i] == dp && q[i] < p))) blocked = true;
        }
      }
    }
    // the group stops at its first kept or blocking neighbour: either way p
    // cannot be kept now, and a position left undecided is decided later
    if ((__ballot(kept_nb || blocked) >> gshift) & gmask) break;
  }
  const bool any_kept = ((__ballot(kept_nb) >> gshift) & gmask) != 0;
  const bool any_blocked = ((__ballot(blocked) >> gshift) & gmask) != 0;
  if (any_kept) {
    if (gl == 0) store_flag(&state[p], kStateAbsorbed);
    return false;
  }
  if (!any_blocked) {
    if (gl == 0) store_flag(&state[p], kStateKept);
    return false;
  }
  return true;
}

constexpr int kVisitLanes = 16;                       // lanes per position in the grid passes
constexpr int kVisitPerBlock = 256 / kVisitLanes;     // positions per 256-thread block

// Bucket offsets of the current call in LDS (E <= 64).
__device__ __forceinline__ void load_offsets(const int32_t* __restrict__ offsets, int E, int* soff) {
  if (threadIdx.x <= static_cast<unsigned>(E)) soff[threadIdx.x] = offsets[threadIdx.x];
  __syncthreads();
}

// One round over all positions (16 lanes each); decided positions return
// at once.  Round 0 also publishes the degrees.
__global__ __launch_bounds__(256) void greedy_round_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state, int r, int32_t* __restrict__ degree_out) {
  __shared__ int soff[kMaxExperts + 1];
  if (*err) return;
  load_offsets(offsets, E, soff);
  const int p = blockIdx.x * kVisitPerBlock + (threadIdx.x / kVisitLanes);
  const int gl = threadIdx.x & (kVisitLanes - 1);
  if (p >= soff[E]) return;
  if (r == 0 && degree_out && gl == 0) degree_out[p] = deg[p];
  if (state[p] != kStateUndecided) return;
  const int e = bucket_of(soff, E, p);
  const int lo = soff[e], n = soff[e + 1] - lo, W = (n + 63) / 64;
  greedy_visit<false, kVisitLanes>(p, lo, n, W, bitmask + bm_off[e] + static_cast<long long>(p - lo) * W, deg,
                                   state);
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
  // coalesced check first: most buckets are fully decided by the grid rounds
  int any = 0;
  for (int i = threadIdx.x; i < n; i += 1024) any |= state[lo + i] == kStateUndecided;
  if (!__syncthreads_or(any)) return;
  const int wv = threadIdx.x >> 6;
  for (int it = 0; it <= n; ++it) {
    int undecided = 0;
    for (int pl = wv; pl < n; pl += 16) {
      const int p = lo + pl;
      if (load_flag(&state[p]) != kStateUndecided) continue;
      if (greedy_visit<true, 64>(p, lo, n, W, bitmask + bm_off[e] + static_cast<long long>(pl) * W, deg, state))
        undecided = 1;
    }
    if (!__syncthreads_or(undecided)) break;
  }
}

// Each kept position offers itself to every neighbour: claim[b] keeps the
// largest key (degree << 32 | ~position), i.e. the neighbour's first kept
// neighbour in walk order.  Only kept positions scan their rows (16 lanes
// each).
__global__ __launch_bounds__(256) void claim_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, const int32_t* __restrict__ state,
    unsigned long long* __restrict__ claim) {
  __shared__ int soff[kMaxExperts + 1];
  if (*err) return;
  load_offsets(offsets, E, soff);
  const int q = blockIdx.x * kVisitPerBlock + (threadIdx.x / kVisitLanes);
  const int gl = threadIdx.x & (kVisitLanes - 1);
  if (q >= soff[E] || state[q] != kStateKept) return;
  const int e = bucket_of(soff, E, q);
  const int lo = soff[e], n = soff[e + 1] - lo, W = (n + 63) / 64;
  const uint64_t* row = bitmask + bm_off[e] + static_cast<long long>(q - lo) * W;
  const unsigned long long key = (static_cast<unsigned long long>(deg[q]) << 32) |
                                 static_cast<unsigned int>(~static_cast<unsigned int>(q));
  for (int wd0 = gl; wd0 < W; wd0 += 4 * kVisitLanes) {
    uint64_t wv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) wv[u] = wd0 + kVisitLanes * u < W ? row[wd0 + kVisitLanes * u] : 0ull;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint64_t bits = wv[u];
      const int cbase = (wd0 + kVisitLanes * u) * 64;
      while (bits) {
        const int b = __ffsll(static_cast<long long>(bits)) - 1;
        bits &= bits - 1;
        if (cbase + b < n) atomicMax(&claim[lo + cbase + b], key);
      }
    }
  }
}

// Representative rows, in two passes over 1024-position blocks.
// rep_local_kernel: the duplicate->representative map, then the rank of each
// representative inside its block (wave ballots + LDS prefix of the 16 wave
// counts) and the block's count.
__global__ __launch_bounds__(1024) void rep_local_kernel(const int32_t* __restrict__ offsets, int E,
                                                        const int* __restrict__ err,
                                                        const int32_t* __restrict__ state,
                                                        const unsigned long long* __restrict__ claim,
                                                        int32_t* __restrict__ rep_of_pos,
                                                        int32_t* __restrict__ local,
                                                        int32_t* __restrict__ bsum, int slot_cap) {
  __shared__ int wcnt[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int p = blockIdx.x * 1024 + tid;
  // state and claim of this position are read together with the slot count
  // (positions past the arrays' T*k entries read nothing)
  const bool mine = p < slot_cap;
  const int st = mine ? state[p] : 0;
  const unsigned long long cl = mine ? claim[p] : 0ull;
  const int failed = *err;
  const int S = offsets[E];
  const int base = blockIdx.x * 1024;
  if (base >= S) return;
  // rep_of_pos: absorbed -> claimed representative; otherwise itself (also
  // after a layout error, when nothing was decided)
  bool f = false;
  if (p < S) {
    const bool absorbed = !failed && st == kStateAbsorbed;
    rep_of_pos[p] = absorbed ? static_cast<int>(~static_cast<unsigned int>(cl & 0xffffffffull)) : p;
    f = !absorbed;
  }
  const uint64_t bal = __ballot(f);
  if (lane == 0) wcnt[wv] = __popcll(bal);
  __syncthreads();
  int before = 0, total = 0;
  for (int i = 0; i < 16; ++i) {
    const int v = wcnt[i];
    before += i < wv ? v : 0;
    total += v;
  }
  if (p < S) local[p] = before + __popcll(bal & lanemask_lt());
  if (tid == 0) bsum[blockIdx.x] = total;
}

// rep_finalize_kernel: every block prefixes the block counts in LDS, then
// writes rep_token, rep_row (through the representative's own block prefix)
// and, in block 0, rep_offsets.
__global__ __launch_bounds__(1024) void rep_finalize_kernel(
    const int32_t* __restrict__ offsets, int E, const int32_t* __restrict__ rep_of_pos,
    const int32_t* __restrict__ perm_token, const int32_t* __restrict__ local,
    const int32_t* __restrict__ bsum, int32_t* __restrict__ rep_row, int32_t* __restrict__ rep_token,
    int32_t* __restrict__ rep_offsets, int slot_cap) {
  extern __shared__ int bpre[];   // one entry per block of the grid, plus one
  __shared__ int wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // this thread's position: its representative and token are read before
  // the block-count scan (positions past the arrays' T*k entries read
  // nothing; those past the kept slot count are read and not used)
  const int p = blockIdx.x * 1024 + tid;
  const bool mine = p < slot_cap;
  const int q_pre = mine ? rep_of_pos[p] : 0;
  const int tok_pre = mine ? perm_token[p] : 0;
  const int S = offsets[E];
  const int nb = (S + 1023) / 1024;
  // exclusive prefix of bsum[0..nb) into bpre, 1024 at a time
  int carry = 0;
  for (int c0 = 0; c0 < nb; c0 += 1024) {
    const int i = c0 + tid;
    const int v = i < nb ? bsum[i] : 0;
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o, 64);
      if (lane >= o) incl += u;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int wb = 0, tot = 0;
    for (int k = 0; k < 16; ++k) {
      wb += k < wv ? wsum[k] : 0;
      tot += wsum[k];
    }
    if (i < nb) bpre[i] = carry + wb + incl - v;
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) bpre[nb] = carry;
  __syncthreads();
  if (p < S) {
    const int q = q_pre;
    const int row = bpre[q >> 10] + local[q];
    rep_row[p] = row;
    if (q == p) rep_token[row] = tok_pre;
  }
  if (blockIdx.x == 0 && tid <= E) {
    const int o = offsets[tid];
    rep_offsets[tid] = o < S ? bpre[o >> 10] + local[o] : bpre[nb];
  }
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
  unsigned long long* claim;
  int32_t* local;
  int32_t* bsum;
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
  w.claim = c.take<unsigned long long>(S);
  w.local = c.take<int32_t>(S);
  w.bsum = c.take<int32_t>((S + 1023) / 1024 + 1);
  w.cap_words = S * ((static_cast<long long>(max_bucket) + 63) / 64);
  w.bitmask = c.take<uint64_t>(static_cast<size_t>(w.cap_words));
  return w;
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
                              void* x_rep, int32_t* degree, const float* inv_norm,
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
  if (d > 32768) return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: d=%d > 32768", d);
  if (static_cast<long long>(T) * d * elem_bytes(dtype) > 0xFFFF0000ll)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: x exceeds 4 GiB - 64 KiB");
  if (static_cast<long long>(T) * k > (1ll << 24))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_condense: T*k > 2^24");
  const size_t need = luffy_condense_workspace_size(T, d, E, k, max_bucket);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_condense: workspace needs %zu bytes, 256-aligned", need);

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  CondenseWs ws = carve_condense(c, T, E, k, max_bucket);
  const int S = T * k;
  const bool bf16 = dtype == LUFFY_BF16;

  // norms from the caller when given (the gate pass already read x)
  const float* inv_norm_use = inv_norm ? inv_norm : ws.inv_norm;
  const int norm_blocks = inv_norm ? std::max(1, (S + 255) / 256) : (T + 3) / 4;
  {
    const int tile = bf16 ? kTile : kTileF32;
#define LUFFY_NORM_ARGS x, T, d, ws.inv_norm, S, ws.deg, ws.state, ws.claim, offsets, E, max_bucket, tile, \
                        ws.cap_words, ws.tile_off, ws.bm_off, ws.err
    if (bf16) {
      if (inv_norm) launch("norm", norm_kernel<true, false>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
      else launch("norm", norm_kernel<true, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
    } else {
      if (inv_norm) launch("norm", norm_kernel<false, false>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
      else launch("norm", norm_kernel<false, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
    }
#undef LUFFY_NORM_ARGS
  }
  {
    if (bf16)
      launch("gram", gram_kernel_bf16, persistent_grid(), GramGemm::THREADS, 0, s, static_cast<const uint16_t*>(x),
             d, perm_token, offsets, E, inv_norm_use, threshold, ws.tile_off, ws.bm_off, ws.err, ws.bitmask,
             ws.deg);
    else
      launch("gram", gram_kernel_f32, 2 * persistent_grid(), 256, 0, s, static_cast<const float*>(x), d, perm_token,
             offsets, E, inv_norm_use, threshold, ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg);
  }
  const int wave_blocks = (S + 3) / 4;
  const int visit_blocks = (S + kVisitPerBlock - 1) / kVisitPerBlock;
  for (int r = 0; r < kGreedyGridRounds; ++r) {
    launch("greedy_round", greedy_round_kernel, visit_blocks, 256, 0, s, offsets, E, ws.bm_off, ws.err, ws.bitmask,
           ws.deg, ws.state, r, degree);
  }
  {
    launch("greedy_finish", greedy_finish_kernel, E, 1024, 0, s, offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg,
           ws.state);
  }
  {
    launch("claim", claim_kernel, visit_blocks, 256, 0, s, offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg,
           ws.state, ws.claim);
  }
  const int pos_blocks = (S + 1023) / 1024;
  {
    launch("rep_local", rep_local_kernel, pos_blocks, 1024, 0, s, offsets, E, ws.err, ws.state, ws.claim,
           rep_of_pos, ws.local, ws.bsum, S);
  }
  {
    launch("rep_finalize", rep_finalize_kernel, pos_blocks, 1024, (pos_blocks + 1) * sizeof(int), s, offsets, E,
           rep_of_pos, perm_token, ws.local, ws.bsum, rep_row, rep_token, rep_offsets, S);
  }
  if (x_rep) {
    launch("gather", gather_kernel, wave_blocks, 256, 0, s, static_cast<const uint8_t*>(x),
           static_cast<size_t>(d) * elem_bytes(dtype), rep_offsets, E, rep_token, static_cast<uint8_t*>(x_rep));
  }
  return check_launch("luffy_condense");
}
