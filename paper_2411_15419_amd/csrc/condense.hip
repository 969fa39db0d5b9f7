// luffy_condense: per-bucket cosine threshold graph, representative
// selection and compaction.
//
// Kernels, in launch order:
//   norm_kernel          1/|x_t| per token (one wave per row); clears the
//                        degree counters and walk states; its first wave
//                        lays out every bucket's tiles and bitmask.
//   gram_kernel_{bf16,f32}  persistent loop over the upper-triangle tiles
//                        (256 rows bf16, 64 rows fp32) of every bucket's Gram
//                        matrix.  The epilogue turns cos >= h into adjacency
//                        bits, writes both the tile and its transpose (every
//                        bitmask word is written exactly once) and adds each
//                        row's edge count to its degree.
//   greedy_round_kernel  first round of the parallel form of the greedy
//                        walk, 16 lanes per position: keeps every position
//                        with no undecided neighbour of higher priority.
//                        A position is claimed by its neighbours as soon
//                        as it is kept, in every pass: it absorbs them and
//                        offers itself (64-bit atomic max of degree,
//                        ~position), so an absorbed position ends with its
//                        first-visited kept neighbour.  On a union of
//                        cliques this round decides every position.
//   greedy_more_kernel   persistent pass with bounded coherent revisits of
//                        positions still undecided (dependency chains).
//   greedy_finish_kernel one workgroup per bucket: a few rounds, then one
//                        visit per position left in priority order (only
//                        when the pass before left a position undecided).
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
#include <atomic>

#include "gemm_core.h"
#include "luffy_common.h"

namespace luffy {
namespace {

constexpr int kGreedyPasses = 32;   // visits of a blocked position in the round after the grid rounds
constexpr int kTile = 256;      // similarity tile of the bf16 path (GramGemm)
constexpr int kTileF32 = 64;    // similarity tile of the fp32 path
constexpr int kGroupsF32 = kTileF32 / 16;   // 16-column bit groups per tile row
constexpr int kWordsF32 = kTileF32 / 64;    // bitmask words per tile row
constexpr int kStateUndecided = 0, kStateKept = 1, kStateAbsorbed = 2;
constexpr int kTileQueues = 8;  // tile queues of the history similarity kernel, one per XCD

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

// fp8 copy of the token rows for the similarity screen (Sec. 3's cosine,
// estimated): row t is normalised and scaled by 2^8, x_n = x * inv_norm[t] *
// 256 (|x_n| = 256 up to the rounding of the norm, every value within
// +-256, inside the E4M3 range), rounded to E4M3 by the hardware conversion
// (values below the smallest normal, 2^-6, stored as 0, so no subnormal
// reaches the MFMA).  rho[t] = |x_n - x^| / |x_n| is taken from the decoded
// bytes, i.e. from the values the MFMA multiplies, and enlarged by 2^-9 to
// cover the float32 sums.  Then for every pair c~ = x^_a . x^_b / 2^16 (the
// raw fp8 product scaled by a power of two) and the cosine c of the bf16
// pass satisfy
//   |c - c~| <= (|x^_a| |e_b| + |e_a| |x_b|) / (|x_a| |x_b|) <= rho_a + rho_b + rho_a rho_b
// (e = x_n - x^, |x_n| = 256), up to float32 rounding.  Row T of x8 (the
// pad row of partial tiles) is zero.  One wave a row (norm_kernel's QUANT
// pass); d % 8 == 0.
__device__ __forceinline__ void gram_quant_row(const uint16_t* __restrict__ x, int T, int d, int t, float inv,
                                               uint8_t* __restrict__ x8, float* __restrict__ rho) {
  const int lane = threadIdx.x & 63;
  uint8_t* out = x8 + static_cast<size_t>(t) * d;
  if (t == T) {
    for (int c = lane * 8; c < d; c += 512) *reinterpret_cast<uint2*>(out + c) = make_uint2(0u, 0u);
    return;
  }
  const uint16_t* row = x + static_cast<size_t>(t) * d;
  const float sc = inv * 256.f;
  float se = 0.f, sx = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    Pack16 v;
    v.u4 = *reinterpret_cast<const uint4*>(row + c);
    float f[8], g[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      f[i] = bf16_to_f32(v.h[i]) * sc;
      g[i] = fabsf(f[i]) < 0x1p-6f ? 0.f : f[i];
    }
    int lo = __builtin_amdgcn_cvt_pk_fp8_f32(g[0], g[1], 0, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(g[2], g[3], lo, true);
    int hi = __builtin_amdgcn_cvt_pk_fp8_f32(g[4], g[5], 0, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(g[6], g[7], hi, true);
    *reinterpret_cast<uint2*>(out + c) = make_uint2(static_cast<uint32_t>(lo), static_cast<uint32_t>(hi));
    const float dq[8] = {__builtin_amdgcn_cvt_f32_fp8(lo, 0), __builtin_amdgcn_cvt_f32_fp8(lo, 1),
                         __builtin_amdgcn_cvt_f32_fp8(lo, 2), __builtin_amdgcn_cvt_f32_fp8(lo, 3),
                         __builtin_amdgcn_cvt_f32_fp8(hi, 0), __builtin_amdgcn_cvt_f32_fp8(hi, 1),
                         __builtin_amdgcn_cvt_f32_fp8(hi, 2), __builtin_amdgcn_cvt_f32_fp8(hi, 3)};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float df = f[i] - dq[i];
      se = fmaf(df, df, se);
      sx = fmaf(f[i], f[i], sx);
    }
  }
  se = wave_sum_f32(se);
  sx = wave_sum_f32(sx);
  if (lane == 0) rho[t] = sx > 0.f ? sqrtf(se / sx) * (1.f + 0x1p-9f) : 0.f;
}

// NORMS = false: the norms were computed by the caller (luffy_route); only
// the clearing and the layout run.  QUANT (bf16): also the similarity
// screen's fp8 rows (gram_quant_row; rows 0..T, T the zero pad row).
template <bool BF16, bool NORMS, bool QUANT = false>
__global__ __launch_bounds__(256) void norm_kernel(const void* __restrict__ xv, int T, int d,
                                                   float* __restrict__ inv_norm, int S,
                                                   int32_t* __restrict__ deg, int32_t* __restrict__ state,
                                                   unsigned long long* __restrict__ claim,
                                                   const int32_t* __restrict__ offsets, int E, int max_bucket,
                                                   int tile, long long cap_words, int32_t* __restrict__ tile_off,
                                                   long long* __restrict__ bm_off, int* __restrict__ err,
                                                   unsigned long long* __restrict__ stats, int* __restrict__ queue,
                                                   int* __restrict__ left, int* __restrict__ list_count,
                                                   uint8_t* __restrict__ x8, float* __restrict__ rho) {
  if (blockIdx.x == 0 && threadIdx.x < 64)
    gram_layout(offsets, E, max_bucket, tile, cap_words, tile_off, bm_off, err);
  if (stats && blockIdx.x == 0 && threadIdx.x >= 64 && threadIdx.x < 68) stats[threadIdx.x - 64] = 0ull;
  if (queue && blockIdx.x == 0 && threadIdx.x >= 128 && threadIdx.x < 128 + kTileQueues) queue[threadIdx.x - 128] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 192) *left = 0;
  // the similarity screen's count of listed tiles
  if (list_count && blockIdx.x == 0 && threadIdx.x == 200) *list_count = 0;
  // also clears the degree counters, walk states and claim keys of all S positions
  for (int p = blockIdx.x * 256 + threadIdx.x; p < S; p += gridDim.x * 256) {
    deg[p] = 0;
    state[p] = 0;
    claim[p] = 0ull;
  }
  if constexpr (!NORMS && !QUANT) return;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if constexpr (QUANT) {
    static_assert(BF16, "fp8 rows of bf16 tokens");
    if (t == T) gram_quant_row(static_cast<const uint16_t*>(xv), T, d, t, 0.f, x8, rho);
    if (t >= T) return;
    if constexpr (!NORMS) {
      gram_quant_row(static_cast<const uint16_t*>(xv), T, d, t, inv_norm[t], x8, rho);
      return;
    }
  }
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
  const float inv = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
  if (lane == 0) inv_norm[t] = inv;
  if constexpr (QUANT) gram_quant_row(static_cast<const uint16_t*>(xv), T, d, t, inv, x8, rho);
}

struct TileCoord {
  int e, ti, tj, lo, n, W;
};

// Bucket of tile `tile` (the last e with tile_off[e] <= tile, skipping
// empty buckets), its first tile, first slot and size.  One load per lane
// (lane e holds bucket e, E <= 64) and a ballot: a single round trip instead
// of a walk of dependent loads.  Called by whole waves.  The _from form
// takes the three per-lane values already loaded (bucket_lookup_loads).
__device__ __forceinline__ void bucket_lookup_loads(const int32_t* __restrict__ tile_off,
                                                    const int32_t* __restrict__ offsets, int E, int& to, int& o0,
                                                    int& o1) {
  const int lane = threadIdx.x & 63;
  const bool in = lane < E;
  to = in ? tile_off[lane] : 0;
  o0 = in ? offsets[lane] : 0;
  o1 = in ? offsets[lane + 1] : 0;
}

__device__ __forceinline__ void locate_bucket_from(int tile, int to, int o0, int o1, int E, int& e, int& tbase,
                                                   int& lo, int& n) {
  const int lane = threadIdx.x & 63;
  const bool in = lane < E;
  e = __popcll(__ballot(in && lane >= 1 && to <= tile));
  tbase = __builtin_amdgcn_readfirstlane(__shfl(to, e, 64));
  lo = __builtin_amdgcn_readfirstlane(__shfl(o0, e, 64));
  n = __builtin_amdgcn_readfirstlane(__shfl(o1, e, 64)) - lo;
}

__device__ __forceinline__ void locate_bucket(int tile, const int32_t* __restrict__ tile_off,
                                              const int32_t* __restrict__ offsets, int E, int& e, int& tbase,
                                              int& lo, int& n) {
  int to, o0, o1;
  bucket_lookup_loads(tile_off, offsets, E, to, o0, o1);
  locate_bucket_from(tile, to, o0, o1, E, e, tbase, lo, n);
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
__device__ __forceinline__ TileCoord decode_tile_grouped_from(int tile, int to, int o0, int o1, int E) {
  TileCoord c;
  int tbase;
  locate_bucket_from(tile, to, o0, o1, E, c.e, tbase, c.lo, c.n);
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

__device__ __forceinline__ TileCoord decode_tile_grouped(int tile, const int32_t* __restrict__ tile_off,
                                                         const int32_t* __restrict__ offsets, int E) {
  int to, o0, o1;
  bucket_lookup_loads(tile_off, offsets, E, to, o0, o1);
  return decode_tile_grouped_from(tile, to, o0, o1, E);
}

// v_writelane_b32: `old` with lane `lane` replaced by the wave-uniform
// `value` (the LLVM intrinsic, which clang does not expose as a builtin).
__device__ int amdgcn_writelane(int value, int lane, int old) __asm("llvm.amdgcn.writelane");

using GramGemm = GemmBig64;
static_assert(GramGemm::BM == kTile && GramGemm::BN == kTile, "similarity tile");


// Tokens of a tile's DMA rows (P rows of tile-row ti, Q rows of tile-row
// tj; rows past the bucket repeat its last row and are not fetched) and the
// tokens whose inverse norms this thread stages for the epilogue: entry i
// of the tile's 2*kTile (P rows, then Q rows) goes to thread i % THREADS,
// as its (i / THREADS)-th (-1 past the bucket).
template <class G>
// pad >= 0: rows past the bucket read row `pad` instead (a zero row, so
// that every fetched row is defined).
__device__ __forceinline__ void gram_tile_tokens(const TileCoord& c, const int32_t* __restrict__ perm_token,
                                                 int32_t (&ptok)[G::LP], int32_t (&qtok)[G::LQ],
                                                 int32_t (&itok)[2 * kTile / G::THREADS], int pad = -1) {
  static_assert((2 * kTile) % G::THREADS == 0, "inverse norms per thread");
  const int32_t* pt = perm_token + c.lo;
#pragma unroll
  for (int j = 0; j < G::LP; ++j) {
    const int r = c.ti * kTile + G::load_row(j);
    ptok[j] = pad >= 0 && r >= c.n ? pad : pt[min(r, c.n - 1)];
  }
#pragma unroll
  for (int j = 0; j < G::LQ; ++j) {
    const int r = c.tj * kTile + G::load_row(G::LP + j) - G::BM;
    qtok[j] = pad >= 0 && r >= c.n ? pad : pt[min(r, c.n - 1)];
  }
#pragma unroll
  for (int u = 0; u < 2 * kTile / G::THREADS; ++u) {
    const int i = static_cast<int>(threadIdx.x) + u * G::THREADS;
    const int r = i < kTile ? c.ti * kTile + i : c.tj * kTile + i - kTile;
    itok[u] = r < c.n ? pt[r] : -1;
  }
}

// Inverse norm staged for the epilogue: NaN for a row outside the bucket,
// which fails every comparison.
__device__ __forceinline__ float gram_stage_inv(const float* __restrict__ inv_norm, int32_t itok) {
  return itok >= 0 ? inv_norm[itok] : __builtin_nanf("");
}

// bits * 2 + (p >= h): the comparison's bit shifted in through the carry
// (an ordered compare: a NaN p shifts in 0).  A VALU read of VCC needs two
// wait states after the VALU write of it: the _next form fills them with the
// next element's product q = (a * b) * c, the last form with a nop.
__device__ __forceinline__ uint32_t shift_in_ge_next(uint32_t bits, float p, float h, float a, float b, float c,
                                                     float& q) {
  asm("v_cmp_le_f32 vcc, %3, %2\n\t"
      "v_mul_f32 %1, %4, %5\n\t"
      "v_mul_f32 %1, %6, %1\n\t"
      "v_addc_co_u32 %0, vcc, %0, %0, vcc"
      : "+v"(bits), "=&v"(q)
      : "v"(p), "s"(h), "v"(a), "v"(b), "v"(c)
      : "vcc");
  return bits;
}

// bits * 2 + (p >= h) and m = min(m, |h - p|) (a NaN p shifts in 0 and
// leaves m): the subtraction and the minimum fill the two wait states of
// the VCC read.
__device__ __forceinline__ uint32_t shift_in_ge_band(uint32_t bits, float p, float h, float& m) {
  float dif;
  asm("v_cmp_le_f32 vcc, %4, %3\n\t"
      "v_sub_f32 %2, %4, %3\n\t"
      "v_min_f32 %1, %1, |%2|\n\t"
      "v_addc_co_u32 %0, vcc, %0, %0, vcc"
      : "+v"(bits), "+v"(m), "=&v"(dif)
      : "v"(p), "s"(h)
      : "vcc");
  return bits;
}

__device__ __forceinline__ uint32_t shift_in_ge_last(uint32_t bits, float p, float h) {
  asm("v_cmp_le_f32 vcc, %2, %1\n\t"
      "s_nop 1\n\t"
      "v_addc_co_u32 %0, vcc, %0, %0, vcc"
      : "+v"(bits)
      : "v"(p), "s"(h)
      : "vcc");
  return bits;
}

// One step of the 32 x 32 bit transpose below: lanes i and i ^ S of a
// half-wave trade the S-bit fields in which bit S of the lane index and of
// the bit index differ.
template <int S>
__device__ __forceinline__ uint32_t transpose_step(uint32_t x, int i) {
  constexpr uint32_t m0 = S == 16 ? 0x0000FFFFu : S == 8 ? 0x00FF00FFu : S == 4 ? 0x0F0F0F0Fu
                        : S == 2 ? 0x33333333u : 0x55555555u;   // bits j with bit S of j clear
  // ds_swizzle bit mode within 32 lanes: and-mask 31, xor-mask S
  const uint32_t y = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(x), 0x1F | (S << 10)));
  const bool up = (i & S) != 0;
  // lower lane: the partner's m0 fields move up by S; upper lane: its ~m0 fields move down by S
  const uint32_t t = __builtin_amdgcn_alignbit(y, y, up ? S : 32 - S);
  const uint32_t keep = up ? ~m0 : m0;
  return (x & keep) | (t & ~keep);
}

// 32 x 32 bit transpose within each half-wave: lane c holds word c of a
// square bit matrix (bit j: entry (j, c)); afterwards lane j holds the word
// with bit c = entry (j, c).
__device__ __forceinline__ uint32_t transpose32_bits(uint32_t x) {
  const int i = opaque_tid() & 31;   // per-lane masks recomputed here, not hoisted out of the tile loop
  x = transpose_step<16>(x, i);
  x = transpose_step<8>(x, i);
  x = transpose_step<4>(x, i);
  x = transpose_step<2>(x, i);
  return transpose_step<1>(x, i);
}

// Modes of the bf16 similarity kernel: every tile on bf16 MFMA; every tile
// on fp8 MFMA as a screen; the bf16 pass over the tiles the screen left.
enum GramMode { kGramPlain = 0, kGramScreen = 1, kGramList = 2 };

// Persistent over the upper-triangle tiles of every bucket.  The loop is
// software-pipelined across tiles: the next tile's bucket lookup is loaded
// before the current tile's K loop (nothing waits on it until the loop is
// over, so it does not hold up the loop's first stages, which the in-order
// load counter would otherwise tie to it); right after the K loop the next
// tile's row tokens are loaded, their latency hidden by this tile's
// compares, and its first DMA stages are issued before the rest of this
// tile's epilogue, which therefore keeps its bit pieces outside the operand
// ring.
//
// kGramScreen (h > 0): X holds the fp8 rows (E4M3 unit rows scaled by 2^8,
// rows of d_units 16-bit units; row T_pad is zero and stands in for the
// rows past a bucket), so a tile's products are 2^16 c~, estimates of the
// cosines with |c~ - c| <= band for every pair: band = 2 r + r^2 + 4e-3, r
// the largest rho (quantisation error, see gram_quant_row) of the
// tile's rows, the constant room for the float32 rounding of both passes.
// A tile whose every value lies outside (h - band, h + band) is decided
// exactly by c~ >= h: it is written as in the bf16 pass.  Any other tile is
// appended to `list` (count in list_count) and leaves its words and degrees
// to the kGramList pass, which recomputes it from the bf16 rows.
template <int MODE>
__global__ __launch_bounds__(GramGemm::THREADS) void gram_kernel_bf16(
    const uint16_t* __restrict__ X, int d_units, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, float h,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg,
    const float* __restrict__ rho, int* __restrict__ list, int* __restrict__ list_count, int T_pad) {
  using G = std::conditional_t<MODE == kGramScreen, GemmBig64F8, GramGemm>;
  static_assert(G::BM == kTile && G::BN == kTile && G::THREADS == GramGemm::THREADS, "similarity tile");
  constexpr int NI = 2 * kTile / G::THREADS;   // inverse norms staged per thread
  static_assert(G::FN % 2 == 0, "column blocks are transposed in pairs");
  // One LDS array: the operand ring, then the inverse norms of the tile's P
  // rows (0..kTile-1) and Q rows (kTile..), then the tile's adjacency
  // pieces, dbits[row][32-column group] and tbits[column][32-row group],
  // then the screen's flag.  With separate LDS variables the compiler loses
  // the alias scopes that tell a stage's fragment reads from the DMA into
  // the other stage, and waits for each stage's DMA right after issuing it
  // (no overlap).
  constexpr int kInvOff = G::LDS_BYTES, kBitsOff = kInvOff + 2 * kTile * 4;
  constexpr int kRhoOff = kBitsOff + 2 * kTile * (kTile / 32) * 4;
  constexpr int kFlagOff = kRhoOff + (MODE == kGramScreen ? 2 * kTile * 4 : 0);
  __shared__ __attribute__((aligned(16))) uint8_t lds[kFlagOff + 16];
  float* rho_ab = reinterpret_cast<float*>(lds + kRhoOff);   // the screen's rho of the P and Q rows
  float* inv_ab = reinterpret_cast<float*>(lds + kInvOff);
  uint32_t (*dbits)[kTile / 32] = reinterpret_cast<uint32_t (*)[kTile / 32]>(lds + kBitsOff);
  uint32_t (*tbits)[kTile / 32] = reinterpret_cast<uint32_t (*)[kTile / 32]>(lds + kBitsOff + kTile * (kTile / 32) * 4);
  int* flag = reinterpret_cast<int*>(lds + kFlagOff);
  const float* inv_a = inv_ab;
  const float* inv_b = inv_ab + kTile;
  if (*err) return;
  const int w = G::wave();
  const int wm = G::wave_m(w), wn = G::wave_n(w);
  // items: tiles 0..total-1, or the listed ones
  const int total = MODE == kGramList ? *list_count : tile_off[E];
  auto tile_of = [&](int item) { return MODE == kGramList ? list[item] : item; };
  int item = xcd_virtual_block();
  if (item >= total) return;   // block-uniform, before any barrier
  int tile = tile_of(item);
  TileCoord c = decode_tile_grouped(tile, tile_off, offsets, E);
  int32_t ptok[G::LP], qtok[G::LQ], itok[NI];
  uint32_t poff[G::LP], qoff[G::LQ];
  // the screen's rows past the bucket read the zero row T (x8 has T + 1)
  constexpr bool SCR = MODE == kGramScreen;
  const int pad = SCR ? T_pad : -1;
  gram_tile_tokens<G>(c, perm_token, ptok, qtok, itok, pad);
#pragma unroll
  for (int j = 0; j < G::LP; ++j) poff[j] = static_cast<uint32_t>(ptok[j]) * d_units;
#pragma unroll
  for (int j = 0; j < G::LQ; ++j) qoff[j] = static_cast<uint32_t>(qtok[j]) * d_units;
  float inv[NI], rh[NI];
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    if constexpr (SCR) rh[u] = itok[u] >= 0 ? rho[itok[u]] : 0.f;
    else inv[u] = gram_stage_inv(inv_norm, itok[u]);
  }
  typename G::Pipe pipe;
  G::prefetch(X, poff, X, qoff, d_units, SCR ? kTile : c.n - c.ti * kTile, SCR ? kTile : c.n - c.tj * kTile, lds,
              pipe);
  for (;;) {
    if constexpr (!SCR) {
#pragma unroll
      for (int u = 0; u < NI; ++u) inv_ab[opaque_tid() + u * G::THREADS] = inv[u];   // visible after the K loop's first barrier
    } else {
#pragma unroll
      for (int u = 0; u < NI; ++u) rho_ab[opaque_tid() + u * G::THREADS] = rh[u];
      if (opaque_tid() == 0) *flag = 0;   // likewise; every wave read the last tile's flag before the loop's barrier
    }
    const int nitem = item + gridDim.x;
    const int next = nitem < total ? tile_of(nitem) : 0;
    int nto = 0, no0 = 0, no1 = 0;
    if (nitem < total) bucket_lookup_loads(tile_off, offsets, E, nto, no0, no1);
    typename G::Acc acc;
    G::zero(acc);
    G::resume(pipe, lds, acc);   // ends with a barrier: the ring is free
    TileCoord cn = c;
    if (nitem < total) {
      cn = decode_tile_grouped_from(next, nto, no0, no1, E);
      gram_tile_tokens<G>(cn, perm_token, ptok, qtok, itok, pad);
    }
    __builtin_amdgcn_sched_barrier(0);

    // Each (fm, fn) block is 32 x 32.  Lane l holds column bbase + l%32 and,
    // in accumulator v, row abase + rv(v) + 4*(l/32), rv(v) = 8(v/4) + v%4.
    // Each lane shifts its 16 compare bits into a word (accumulator v at bit
    // v) and spreads them to bits rv(v); lanes c and c+32 merge theirs with
    // one cross-half exchange, which gives the column pieces (the mirrored
    // tile's row words).  The row pieces are the bit transposes of the
    // column pieces: the two column blocks of a wave are transposed
    // together, one per half-wave.  Edge test: dot * (1/|a|) * (1/|b|) >= h
    // (rows outside the bucket carry a NaN scale), never a token with
    // itself.  The screen tests its product against 2^16 h (its rows past
    // the bucket are zero: no edge for h > 0) and also keeps the least
    // |product - 2^16 h| of the lane.
    // lane values recomputed from the opaque thread index: hoisted out of
    // the tile loop they would stay live across the K loop
    const int el = opaque_tid() & 63;
    const int l31 = el & 31, hi = el >> 5;
    const bool same_tile = c.ti == c.tj;
    float dmin = __builtin_inff(), band = 0.f;
    if constexpr (MODE == kGramScreen) {
      // |c~ - c| <= rho_a + rho_b + rho_a rho_b over the tile's rows
      float r = 0.f;
#pragma unroll
      for (int q = 0; q < 2 * kTile / 256; ++q) {
        const float4 f = *reinterpret_cast<const float4*>(&rho_ab[256 * q + 4 * el]);
        r = fmaxf(r, fmaxf(fmaxf(f.x, f.y), fmaxf(f.z, f.w)));
      }
      for (int o = 32; o >= 1; o >>= 1) r = fmaxf(r, __shfl_xor(r, o, 64));
      band = (2.f * r + r * r + 4e-3f) * 65536.f;
    }
    const float hs = h * 65536.f;   // the threshold in units of the screen's products (exact)
#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm) {
      const int abase = wm * G::WTM + 32 * fm;
      // this lane's 16 rows: abase + 8q + 4hi + r, as 4 runs of 4
      float ia[16];
      if constexpr (!SCR) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 f = *reinterpret_cast<const float4*>(&inv_a[abase + 8 * q + 4 * hi]);
          ia[4 * q] = f.x;
          ia[4 * q + 1] = f.y;
          ia[4 * q + 2] = f.z;
          ia[4 * q + 3] = f.w;
        }
      }
      uint32_t col[G::FN];
#pragma unroll
      for (int fn = 0; fn < G::FN; ++fn) {
        const int bbase = wn * G::WTN + 32 * fn;
        const int bl = bbase + l31;
        uint32_t bits = 0;
        if constexpr (SCR) {
          // raw fp8 products of unit rows scaled by 2^8: c~ = acc / 2^16;
          // a token with itself is set to 0 (no edge for h > 0, and it
          // stays out of the band; the word drops it below anyway)
          if (same_tile && abase == bbase) {
#pragma unroll
            for (int v = 0; v < 16; ++v)
              if (8 * (v >> 2) + (v & 3) + 4 * hi == l31) acc[fm][fn][v] = 0.f;
          }
          // a 32 x 32 block without an edge (every product below 2^16 h,
          // the common case) needs only its largest product: no bits, and
          // its least distance to 2^16 h is 2^16 h minus that product
          float mx = acc[fm][fn][0];
#pragma unroll
          for (int v = 1; v < 16; ++v) mx = fmaxf(mx, acc[fm][fn][v]);
          if (__ballot(mx >= hs) == 0) {
            dmin = fminf(dmin, hs - mx);
          } else {
#pragma unroll
            for (int v = 15; v >= 0; --v) bits = shift_in_ge_band(bits, acc[fm][fn][v], hs, dmin);
          }
        } else {
          const float ib = inv_b[bl];
          float p = acc[fm][fn][15] * ia[15] * ib;
#pragma unroll
          for (int v = 15; v >= 1; --v) {
            float q;
            bits = shift_in_ge_next(bits, p, h, acc[fm][fn][v - 1], ia[v - 1], ib, q);
            p = q;
          }
          bits = shift_in_ge_last(bits, p, h);
        }
        // nibble k (accumulators 4k..4k+3) to bits 8k..8k+3, then this half's rows
        bits = (bits & 0xFFu) | ((bits & 0xFF00u) << 8);
        bits = (bits & 0x000F000Fu) | ((bits & 0x00F000F0u) << 4);
        bits <<= 4 * hi;
        uint32_t cw = bits | static_cast<uint32_t>(__shfl_xor(static_cast<int>(bits), 32, 64));
        if (same_tile && abase == bbase) cw &= ~(1u << l31);   // the token with itself
        col[fn] = cw;
        if (hi == 0) tbits[bl][abase >> 5] = cw;
      }
#pragma unroll
      for (int p = 0; p < G::FN / 2; ++p) {
        // lower half-wave: block 2p, upper: block 2p + 1 (a select, not an
        // indexed read, which would put col in memory)
        const uint32_t sel = col[2 * p] ^ ((col[2 * p] ^ col[2 * p + 1]) & (0u - static_cast<uint32_t>(hi)));
        const uint32_t rowbits = transpose32_bits(sel);
        dbits[abase + l31][(wn * G::WTN + 32 * (2 * p + hi)) >> 5] = rowbits;
      }
    }
    if constexpr (MODE == kGramScreen) {
      if (__ballot(dmin < band) != 0 && el == 0) *flag = 1;
    }
    __builtin_amdgcn_sched_barrier(0);
    if (nitem < total) {
#pragma unroll
      for (int j = 0; j < G::LP; ++j) poff[j] = static_cast<uint32_t>(ptok[j]) * d_units;
#pragma unroll
      for (int j = 0; j < G::LQ; ++j) qoff[j] = static_cast<uint32_t>(qtok[j]) * d_units;
      // before the DMA: waiting for them then does not wait for the DMA
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        if constexpr (SCR) rh[u] = itok[u] >= 0 ? rho[itok[u]] : 0.f;
        else inv[u] = gram_stage_inv(inv_norm, itok[u]);
      }
      G::prefetch(X, poff, X, qoff, d_units, SCR ? kTile : cn.n - cn.ti * kTile, SCR ? kTile : cn.n - cn.tj * kTile,
                  lds, pipe);
    }
    // LDS-only barriers from here on: a full __syncthreads() would also wait
    // for the next tile's DMA
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's pieces are in LDS
    raw_barrier();
    bool decided = true;
    if constexpr (MODE == kGramScreen) {
      decided = *flag == 0;
      if (!decided && opaque_tid() == 0) list[atomicAdd(list_count, 1)] = tile;
    }
    if (decided) {
      // degree: edges of each tile row (and, off the diagonal, of each mirrored row)
      for (int i = opaque_tid(); i < 2 * kTile; i += G::THREADS) {
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
      for (int i = opaque_tid(); i < kTile * 4; i += G::THREADS) {
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
    }
    if (nitem >= total) break;
    // every wave's reads of the pieces, of inv_ab, rho_ab and the flag are
    // done before the next tile overwrites them
    __builtin_amdgcn_s_waitcnt(0xC07F);
    raw_barrier();
    item = nitem;
    tile = next;
    c = cn;
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

// ------------------------------------------------------------ history
// Historical similarity (Sec. 5.1 step 2): a pair of tokens whose weight in
// the previous block was above S1 takes weight 1 here, one below S2 takes
// weight 0, and only the other pairs use their cosine.  A block leaves the
// next one a record of its own weights as two bit classes per pair of
// positions of one bucket, in the layout of the adjacency bitmask:
// hi (weight > S1) and lo (weight < S2), with hi taking precedence.  The
// record also keeps the block's token -> position map and bucket layout, so
// the next block, whose buckets differ, can find a pair (t, u) in it: the
// pair is decided when t and u shared a bucket there.
constexpr int kHistMagic = 0x4C594831;   // record format tag

struct HistRec {
  int32_t* info;        // magic, T, E, k, max_bucket
  int32_t* slot_pos;    // [T*k] position of slot (t, j) in the writing block, -1 if dropped
  int32_t* offsets;     // [E+1] its buckets
  long long* word_off;  // [E+1] first word of bucket e in hi and lo
  uint64_t* hi;         // [cap_words]
  uint64_t* lo;         // [cap_words]
};

HistRec carve_hist(Carver& c, int T, int E, int k, int max_bucket) {
  HistRec h;
  const long long S = static_cast<long long>(T) * k;
  const long long cap_words = S * ((static_cast<long long>(max_bucket) + 63) / 64);
  h.info = c.take<int32_t>(8);
  h.slot_pos = c.take<int32_t>(static_cast<size_t>(S));
  h.offsets = c.take<int32_t>(E + 1);
  h.word_off = c.take<long long>(E + 1);
  h.hi = c.take<uint64_t>(static_cast<size_t>(cap_words));
  h.lo = c.take<uint64_t>(static_cast<size_t>(cap_words));
  return h;
}


// Header of the record a block leaves: format, sizes, the token -> position
// map, bucket offsets and word offsets (after the layout).  A layout error
// (a bucket larger than max_bucket) leaves the record marked invalid, which
// makes the next block compute every pair.
__global__ __launch_bounds__(256) void hist_header_kernel(const int32_t* __restrict__ slot_pos, int T, int k,
                                                          const int32_t* __restrict__ offsets, int E, int max_bucket,
                                                          const long long* __restrict__ bm_off,
                                                          const int* __restrict__ err, HistRec out) {
  const long long S = static_cast<long long>(T) * k;
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < S; i += gridDim.x * 256ll) out.slot_pos[i] = slot_pos[i];
  if (blockIdx.x == 0) {
    if (threadIdx.x <= static_cast<unsigned>(E)) {
      out.offsets[threadIdx.x] = offsets[threadIdx.x];
      out.word_off[threadIdx.x] = bm_off[threadIdx.x];
    }
    if (threadIdx.x == 0) {
      out.info[0] = *err ? 0 : kHistMagic;
      out.info[1] = T;
      out.info[2] = E;
      out.info[3] = k;
      out.info[4] = max_bucket;
    }
  }
}

// Previous position of every slot of every position of this block, as
// (previous bucket << 24) | position inside it, -1 where the token had no
// kept slot there; every entry -1 when the record does not match (T, E, k,
// max_bucket) or is marked invalid.  One thread per position.
template <int K>
__global__ __launch_bounds__(256) void hist_cols_kernel(const int32_t* __restrict__ offsets, int E,
                                                        const int32_t* __restrict__ perm_token,
                                                        const int* __restrict__ err, HistRec in, int T,
                                                        int max_bucket, int32_t* __restrict__ colinfo) {
  __shared__ int poff[kMaxExperts + 1];
  __shared__ int rec_ok;
  if (*err) return;
  if (threadIdx.x == 0)
    rec_ok = in.info[0] == kHistMagic && in.info[1] == T && in.info[2] == E && in.info[3] == K &&
             in.info[4] == max_bucket;
  __syncthreads();
  const bool ok = rec_ok;
  if (ok && threadIdx.x <= static_cast<unsigned>(E)) poff[threadIdx.x] = in.offsets[threadIdx.x];
  __syncthreads();
  const int S = offsets[E];
  for (int p = blockIdx.x * 256 + threadIdx.x; p < S; p += gridDim.x * 256) {
    const int u = perm_token[p];
#pragma unroll
    for (int j = 0; j < K; ++j) {
      int v = -1;
      if (ok) {
        const int q = in.slot_pos[static_cast<size_t>(u) * K + j];
        if (q >= 0) {
          const int pe = bucket_of(poff, E, q);
          v = (pe << 24) | (q - poff[pe]);
        }
      }
      colinfo[static_cast<size_t>(p) * K + j] = v;
    }
  }
}

// The previous block's classes of every pair of this block's buckets, in
// this block's bitmask layout: rb_hi / rb_lo bit c of row a of bucket e is
// set when tokens perm_token[lo+a] and perm_token[lo+c] shared a bucket in
// the previous block with class hi / lo there.  One block per kGatherRows
// rows of one bucket; each wave walks 64 columns of a 256-column chunk (the
// columns' previous positions from colinfo), and for each row reads the
// previous row's word of each matching column straight from memory (a row is
// a few KB, so its words stay in L1 / L2 while the block walks it).
constexpr int kGatherRows = 8;

template <int K>
__global__ __launch_bounds__(256) void hist_gather_kernel(const int32_t* __restrict__ offsets, int E,
                                                          const long long* __restrict__ bm_off,
                                                          const int* __restrict__ err, HistRec in,
                                                          const int32_t* __restrict__ colinfo,
                                                          uint64_t* __restrict__ rb_hi, uint64_t* __restrict__ rb_lo) {
  __shared__ int rinfo[kGatherRows][K];        // previous bucket of the rows' slots (-1: none)
  __shared__ long long rbase[kGatherRows][K];  // first word of that previous row
  __shared__ int tile_e, tile_a0, tile_rows;
  if (*err) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  constexpr int G = kGatherRows;
  if (w == 0) {
    // this block's bucket and first row: lane e holds bucket e's row groups
    const int n = lane < E ? offsets[lane + 1] - offsets[lane] : 0;
    const int g = (n + G - 1) / G;
    int incl = g;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
    const int b = blockIdx.x;
    const int e = __popcll(__ballot(lane < E && incl <= b));
    const int es = e < E ? e : 0;
    const int excl = __shfl(incl - g, es, 64);
    const int ne = __shfl(n, es, 64);
    if (lane == 0) {
      tile_e = e < E ? e : -1;
      tile_a0 = (b - excl) * G;
      tile_rows = min(G, ne - tile_a0);
    }
  }
  __syncthreads();
  const int e = tile_e;
  if (e < 0) return;
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  const int a0 = tile_a0, rows = tile_rows;
  if (tid < G * K) {
    const int i = tid / K, j = tid % K;
    const int ri = i < rows ? colinfo[static_cast<size_t>(lo + a0 + i) * K + j] : -1;
    long long base = 0;
    if (ri >= 0) {
      const int pe = ri >> 24, pl = ri & 0xFFFFFF;
      const int wq = (in.offsets[pe + 1] - in.offsets[pe] + 63) / 64;
      base = in.word_off[pe] + static_cast<long long>(pl) * wq;
    }
    rinfo[i][j] = ri < 0 ? -1 : (ri >> 24);
    rbase[i][j] = base;
  }
  __syncthreads();
  for (int c0 = 0; c0 < n; c0 += 256) {
    const int c = c0 + tid;
    int qv[K];
#pragma unroll
    for (int j = 0; j < K; ++j) qv[j] = c < n ? colinfo[static_cast<size_t>(lo + c) * K + j] : -1;
    const int wd = (c0 >> 6) + w;
    // the words of all G rows are loaded before any is used, so their
    // latencies overlap
    long long widx[G];
    int bit[G];
#pragma unroll
    for (int i = 0; i < G; ++i) {
      widx[i] = -1;
      bit[i] = 0;
#pragma unroll
      for (int jr = K - 1; jr >= 0; --jr) {
        const int pe = i < rows ? rinfo[i][jr] : -1;
#pragma unroll
        for (int jc = K - 1; jc >= 0; --jc) {
          if (pe >= 0 && qv[jc] >= 0 && (qv[jc] >> 24) == pe) {
            const int q = qv[jc] & 0xFFFFFF;
            widx[i] = rbase[i][jr] + (q >> 6);
            bit[i] = q & 63;
          }
        }
      }
    }
    uint64_t vh[G], vl[G];
#pragma unroll
    for (int i = 0; i < G; ++i) {
      vh[i] = widx[i] >= 0 ? in.hi[widx[i]] : 0ull;
      vl[i] = widx[i] >= 0 ? in.lo[widx[i]] : 0ull;
    }
#pragma unroll
    for (int i = 0; i < G; ++i) {
      if (i >= rows) break;
      const uint64_t mh = __ballot((vh[i] >> bit[i]) & 1ull), ml = __ballot((vl[i] >> bit[i]) & 1ull);
      if (lane == 0 && wd < W) {
        const long long o = bm_off[e] + static_cast<long long>(a0 + i) * W + wd;
        rb_hi[o] = mh;
        rb_lo[o] = ml;
      }
    }
  }
}

// Constants of a block's pair weights: a decided pair's weight is 1 or 0,
// which gives its edge (w >= h) and its classes for the next block
// (w > S1, w < S2) without a cosine.
struct HistParams {
  float h, S1, S2;
  uint64_t* out_hi;   // record words of this block (nullptr: no record)
  uint64_t* out_lo;
  const uint64_t* rb_hi;   // previous classes in this block's layout (nullptr: none)
  const uint64_t* rb_lo;
  unsigned long long* stats;   // undecided pairs, decided pairs, tiles computed, tiles skipped
  int* queue;                  // kTileQueues tile counters, zero at launch
};

// Words of one row piece from its (hi, lo) previous classes, for a tile
// whose pairs are all decided: edge, class hi and class lo of every pair
// under the valid mask vm.
__device__ __forceinline__ void decided_words(uint64_t hi, uint64_t lo, uint64_t vm, const HistParams& hp,
                                              uint64_t& edge, uint64_t& rh, uint64_t& rl) {
  const uint64_t one = hi & vm, zero = lo & ~hi & vm;
  edge = (1.0f >= hp.h ? one : 0ull) | (0.0f >= hp.h ? zero : 0ull);
  rh = (1.0f > hp.S1 ? one : 0ull) | (0.0f > hp.S1 ? zero : 0ull);
  rl = (1.0f < hp.S2 ? one : 0ull) | (0.0f < hp.S2 ? zero : 0ull);
}

// Columns of word wd (global word index) of a row that are pairs inside the
// bucket: columns < n, the row's own position excluded.
__device__ __forceinline__ uint64_t pair_mask(int row, int wd, int n) {
  const int c0 = wd * 64;
  uint64_t m = n - c0 >= 64 ? ~0ull : (n - c0 <= 0 ? 0ull : (1ull << (n - c0)) - 1);
  if (row >= c0 && row < c0 + 64) m &= ~(1ull << (row - c0));
  return m;
}

// bf16 similarity with history.  Per tile: the previous classes of its pairs
// (rows of tile-row ti, words of tile-column tj) are read into LDS; the
// undecided and decided pairs above the diagonal are counted; a tile whose
// pairs are all decided skips the product and derives its words from the
// classes alone (its mirror from the mirrored classes, which are the same
// pairs); any other tile runs the product and takes, pair by pair, weight 1
// or 0 where the previous block decided it and the cosine elsewhere.  The
// record of this block (classes of every weight) is written beside the
// adjacency words, direct and mirrored.
template <bool HIN, bool HOUT>
__global__ __launch_bounds__(GramGemm::THREADS) void gram_hist_kernel_bf16(
    const uint16_t* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, HistParams hp,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg) {
  using G = GramGemm;
  __shared__ __attribute__((aligned(16))) uint8_t lds[G::LDS_BYTES];
  __shared__ __attribute__((aligned(16))) float inv_a[kTile];
  __shared__ float inv_b[kTile];
  __shared__ __attribute__((aligned(16))) uint64_t rbw[2][kTile][4];   // previous classes of the tile's pairs
  __shared__ unsigned long long cnt_s[2];
  constexpr int NM = HOUT ? 3 : 1;   // masks built per tile: edge, then class hi and class lo
  // after the K loop the operand buffers hold the masks' pieces:
  // dbits[m][row][32-column group], tbits[m][column][32-row group]
  auto dbits = reinterpret_cast<uint32_t (*)[kTile][kTile / 32]>(lds);
  auto tbits = reinterpret_cast<uint32_t (*)[kTile][kTile / 32]>(lds + NM * kTile * kTile / 8);
  static_assert(2 * NM * kTile * kTile / 8 <= G::LDS_BYTES, "mask pieces fit the operand buffer");
  if (*err) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = G::wave_m(w), wn = G::wave_n(w);
  const int total = tile_off[E];
  // Tiles cost very different times (skipped or computed), so blocks take
  // them from queues: queue x holds the x-th eighth of the tile order, a
  // block first drains the queue of its own XCD (blocks are dealt to the
  // XCDs round-robin), then the others'.
  __shared__ int next_tile;
  const int home = blockIdx.x % kTileQueues;
  int qi = 0;
  for (;;) {
    if (tid == 0) {
      int t = -1;
      while (qi < kTileQueues) {
        const int x = (home + qi) % kTileQueues;
        const int t0 = static_cast<int>(static_cast<long long>(total) * x / kTileQueues);
        const int t1 = static_cast<int>(static_cast<long long>(total) * (x + 1) / kTileQueues);
        const int v = atomicAdd(&hp.queue[x], 1);
        if (t0 + v < t1) {
          t = t0 + v;
          break;
        }
        ++qi;
      }
      next_tile = t;
    }
    __syncthreads();
    const int tile = next_tile;
    if (tile < 0) break;
    const TileCoord c = decode_tile_grouped(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    const long long bmo = bm_off[c.e];
    const int nrow_a = c.n - c.ti * kTile, nrow_b = c.n - c.tj * kTile;
    const bool same_tile = c.ti == c.tj;
    // previous classes of the tile's pairs; count undecided / decided pairs
    // above the diagonal
    if (tid < 2) cnt_s[tid] = 0;
    __syncthreads();
    int undecided = 0;
    {
      unsigned long long nu = 0, nd = 0;
      for (int i = tid; i < kTile * 4; i += G::THREADS) {
        const int rl = i >> 2, ww = i & 3;
        const int a = c.ti * kTile + rl, wd = 4 * c.tj + ww;
        uint64_t h1 = 0, l1 = 0, vm = 0;
        if (a < c.n && wd < c.W) {
          vm = pair_mask(a, wd, c.n);
          if constexpr (HIN) {
            h1 = hp.rb_hi[bmo + static_cast<long long>(a) * c.W + wd];
            l1 = hp.rb_lo[bmo + static_cast<long long>(a) * c.W + wd];
          }
        }
        rbw[0][rl][ww] = h1;
        rbw[1][rl][ww] = l1;
        const uint64_t und = ~(h1 | l1) & vm;
        undecided |= und != 0;
        // pairs above the diagonal only (columns > row) on a diagonal tile
        uint64_t up = ~0ull;
        if (same_tile) {
          const int c0 = wd * 64;
          up = a < c0 ? ~0ull : (a >= c0 + 63 ? 0ull : ~((2ull << (a - c0)) - 1));
        }
        nu += __popcll(und & up);
        nd += __popcll(vm & ~und & up);
      }
      if (nu) atomicAdd(&cnt_s[0], nu);
      if (nd) atomicAdd(&cnt_s[1], nd);
    }
    undecided = __syncthreads_or(undecided);
    if (tid == 0) {
      atomicAdd(&hp.stats[0], cnt_s[0]);
      atomicAdd(&hp.stats[1], cnt_s[1]);
      atomicAdd(&hp.stats[undecided ? 2 : 3], 1ull);
    }
    if (!undecided) {
      // every pair decided: no product; direct words from rbw, mirrored
      // words from the mirrored classes (same pairs, read from rb)
      for (int i = tid; i < 2 * kTile * 4; i += G::THREADS) {
        const bool mirror = i >= kTile * 4;
        if (mirror && same_tile) continue;
        const int j = mirror ? i - kTile * 4 : i;
        const int rl = j >> 2, ww = j & 3;
        const int a = (mirror ? c.tj : c.ti) * kTile + rl, wd = 4 * (mirror ? c.ti : c.tj) + ww;
        if (a >= c.n || wd >= c.W) continue;
        const long long o = bmo + static_cast<long long>(a) * c.W + wd;
        const uint64_t h1 = mirror ? hp.rb_hi[o] : rbw[0][rl][ww];
        const uint64_t l1 = mirror ? hp.rb_lo[o] : rbw[1][rl][ww];
        uint64_t edge, rh, rlw;
        decided_words(h1, l1, pair_mask(a, wd, c.n), hp, edge, rh, rlw);
        bitmask[o] = edge;
        if constexpr (HOUT) {
          hp.out_hi[o] = rh;
          hp.out_lo[o] = rlw;
        }
        if (edge) atomicAdd(&deg[c.lo + a], __popcll(edge));
      }
      __syncthreads();
      continue;
    }
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
    G::run(X, poff, X, qoff, d, nrow_a, nrow_b, lds, acc);  // ends with a barrier

    // Epilogue as in gram_kernel_bf16, for NM predicates per pair:
    //   weight w = 1 (class hi), 0 (class lo) or the cosine;
    //   edge = w >= h; next classes w > S1, w < S2.
    const int l31 = lane & 31, hi = lane >> 5;
    const uint32_t* rbh32 = reinterpret_cast<const uint32_t*>(&rbw[0][0][0]);
    const uint32_t* rbl32 = reinterpret_cast<const uint32_t*>(&rbw[1][0][0]);
    const bool e1 = 1.0f >= hp.h, e0 = 0.0f >= hp.h;
    const bool h1c = 1.0f > hp.S1, h0c = 0.0f > hp.S1, l1c = 1.0f < hp.S2, l0c = 0.0f < hp.S2;
#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm) {
      const int abase = wm * G::WTM + 32 * fm;
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
        uint32_t colbits[NM], piece[NM];
#pragma unroll
        for (int m = 0; m < NM; ++m) colbits[m] = piece[m] = 0;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int rv = 8 * (v >> 2) + (v & 3);
          const int row = abase + rv + 4 * hi;
          const bool hb = (rbh32[row * 8 + (bbase >> 5)] >> l31) & 1u;
          const bool lb = (rbl32[row * 8 + (bbase >> 5)] >> l31) & 1u;
          const float cs = acc[fm][fn][v] * ia[v] * ib;
          const bool self = diag && rv + 4 * hi == l31;
          bool pr[NM];
          pr[0] = !self && (hb ? e1 : (lb ? e0 : cs >= hp.h));
          if constexpr (HOUT) {
            pr[1] = !self && (hb ? h1c : (lb ? h0c : cs > hp.S1));
            pr[2] = !self && (hb ? l1c : (lb ? l0c : cs < hp.S2));
          }
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            const uint64_t bm = __ballot(pr[m]);
            piece[m] = amdgcn_writelane(static_cast<int>(static_cast<uint32_t>(bm)), rv, piece[m]);
            piece[m] = amdgcn_writelane(static_cast<int>(static_cast<uint32_t>(bm >> 32)), rv + 4, piece[m]);
            colbits[m] |= pr[m] ? 1u << rv : 0u;
          }
        }
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          colbits[m] <<= 4 * hi;
          const uint32_t tv = colbits[m] | static_cast<uint32_t>(__shfl_xor(static_cast<int>(colbits[m]), 32, 64));
          if (lane < 32) {
            dbits[m][abase + l31][bbase >> 5] = piece[m];
            tbits[m][bl][abase >> 5] = tv;
          }
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < 2 * kTile; i += G::THREADS) {
      const bool mirror = i >= kTile;
      const int rl = mirror ? i - kTile : i;
      const uint32_t* pcs = mirror ? tbits[0][rl] : dbits[0][rl];
      int cnt = 0;
#pragma unroll
      for (int g = 0; g < kTile / 32; ++g) cnt += __popc(pcs[g]);
      const int r = (mirror ? c.tj : c.ti) * kTile + rl;
      if (cnt && r < c.n && (!mirror || !same_tile)) atomicAdd(&deg[c.lo + r], cnt);
    }
    for (int i = tid; i < kTile * 4; i += G::THREADS) {
      const int rl = i >> 2, ww = i & 3;
      const int a = c.ti * kTile + rl, wd = 4 * c.tj + ww;
      const int bb = c.tj * kTile + rl, wt = 4 * c.ti + ww;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        uint64_t* dst = m == 0 ? bitmask : (m == 1 ? hp.out_hi : hp.out_lo);
        const uint64_t dv = static_cast<uint64_t>(dbits[m][rl][2 * ww]) |
                            (static_cast<uint64_t>(dbits[m][rl][2 * ww + 1]) << 32);
        if (a < c.n && wd < c.W) dst[bmo + static_cast<long long>(a) * c.W + wd] = dv;
        if (!same_tile) {
          const uint64_t tv = static_cast<uint64_t>(tbits[m][rl][2 * ww]) |
                              (static_cast<uint64_t>(tbits[m][rl][2 * ww + 1]) << 32);
          if (bb < c.n && wt < c.W) dst[bmo + static_cast<long long>(bb) * c.W + wt] = tv;
        }
      }
    }
    __syncthreads();
  }
}

// float32 similarity with history: the 64-row tiles of gram_kernel_f32, every
// tile computed; each pair takes weight 1 or 0 where the previous block
// decided it and its cosine elsewhere; the record words are written beside
// the adjacency words.
template <bool HIN, bool HOUT>
__global__ __launch_bounds__(256) void gram_hist_kernel_f32(
    const float* __restrict__ X, int d, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ offsets, int E, const float* __restrict__ inv_norm, HistParams hp,
    const int32_t* __restrict__ tile_off, const long long* __restrict__ bm_off,
    const int* __restrict__ err, uint64_t* __restrict__ bitmask, int32_t* __restrict__ deg) {
  constexpr int KC = 16;
  constexpr int NM = HOUT ? 3 : 1;
  __shared__ float Ps[kTileF32][KC + 1];
  __shared__ float Qs[kTileF32][KC + 1];
  constexpr int MT = kTileF32 / 16;
  __shared__ uint8_t pred[kTileF32][kTileF32];   // bit m: predicate m of the pair
  __shared__ uint16_t dbits[NM][kTileF32][kGroupsF32];
  __shared__ uint16_t tbits[NM][kTileF32][kGroupsF32];
  __shared__ float inv_a[kTileF32], inv_b[kTileF32];
  __shared__ uint64_t rbw[2][kTileF32];
  if (*err) return;
  const int tid = threadIdx.x;
  const int rb = (tid >> 4) * MT, cb = (tid & 15) * MT;
  const int total = tile_off[E];
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    const TileCoord c = decode_tile(tile, tile_off, offsets, E);
    const int32_t* pt = perm_token + c.lo;
    const long long bmo = bm_off[c.e];
    if (tid < kTileF32) inv_a[tid] = inv_norm[pt[min(c.ti * kTileF32 + tid, c.n - 1)]];
    else if (tid < 2 * kTileF32) inv_b[tid - kTileF32] = inv_norm[pt[min(c.tj * kTileF32 + tid - kTileF32, c.n - 1)]];
    else if (tid < 3 * kTileF32) {
      // previous classes: tile-row rows, word tj (64-column tiles are one word)
      const int rl = tid - 2 * kTileF32, a = c.ti * kTileF32 + rl;
      uint64_t h1 = 0, l1 = 0;
      if constexpr (HIN) {
        if (a < c.n) {
          h1 = hp.rb_hi[bmo + static_cast<long long>(a) * c.W + c.tj];
          l1 = hp.rb_lo[bmo + static_cast<long long>(a) * c.W + c.tj];
        }
      }
      rbw[0][rl] = h1;
      rbw[1][rl] = l1;
    }
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
    unsigned long long nu = 0, nd = 0;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        const int a = c.ti * kTileF32 + rb + i, b = c.tj * kTileF32 + cb + j;
        const bool pair = a < c.n && b < c.n && a != b;
        const bool hb = (rbw[0][rb + i] >> (cb + j)) & 1ull, lb = (rbw[1][rb + i] >> (cb + j)) & 1ull;
        const float cs = acc[i][j] * inv_a[rb + i] * inv_b[cb + j];
        const float wv = hb ? 1.0f : (lb ? 0.0f : cs);
        uint8_t p = 0;
        if (pair) {
          p |= wv >= hp.h ? 1 : 0;
          p |= wv > hp.S1 ? 2 : 0;
          p |= wv < hp.S2 ? 4 : 0;
          if (a < b) {
            if (hb || lb) ++nd;
            else ++nu;
          }
        }
        pred[rb + i][cb + j] = p;
      }
    if (nu) atomicAdd(&hp.stats[0], nu);
    if (nd) atomicAdd(&hp.stats[1], nd);
    if (tid == 0) atomicAdd(&hp.stats[2], 1ull);
    __syncthreads();
    for (int idx = tid; idx < NM * kTileF32 * kGroupsF32; idx += 256) {
      const int m = idx / (kTileF32 * kGroupsF32), rem = idx % (kTileF32 * kGroupsF32);
      const int r = rem / kGroupsF32, g = rem % kGroupsF32;
      uint32_t dv = 0, tv = 0;
      for (int bit = 0; bit < 16; ++bit) {
        dv |= static_cast<uint32_t>((pred[r][16 * g + bit] >> m) & 1) << bit;
        tv |= static_cast<uint32_t>((pred[16 * g + bit][r] >> m) & 1) << bit;
      }
      dbits[m][r][g] = static_cast<uint16_t>(dv);
      tbits[m][r][g] = static_cast<uint16_t>(tv);
    }
    __syncthreads();
    if (tid < 2 * kTileF32) {
      const bool mirror = tid >= kTileF32;
      const int rl = mirror ? tid - kTileF32 : tid;
      int cnt = 0;
      for (int g = 0; g < kGroupsF32; ++g) cnt += __popc(mirror ? tbits[0][rl][g] : dbits[0][rl][g]);
      const int r = (mirror ? c.tj : c.ti) * kTileF32 + rl;
      if (cnt && r < c.n && (!mirror || c.ti != c.tj)) atomicAdd(&deg[c.lo + r], cnt);
    }
    write_tile_words(c, dbits[0], tbits[0], bitmask, bmo);
    if constexpr (HOUT) {
      write_tile_words(c, dbits[1], tbits[1], hp.out_hi, bmo);
      write_tile_words(c, dbits[2], tbits[2], hp.out_lo, bmo);
    }
    __syncthreads();
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
// U words a lane of a GW-lane group, from word b0 of a row on: looks up the
// state and degree of every neighbour they hold and notes a kept
// neighbour or an undecided one of higher priority.
template <bool FRESH, int GW, int U>
__device__ __forceinline__ void greedy_scan(int b0, int p, int dp, int lo, int n, int W,
                                            const uint64_t* __restrict__ row, const int32_t* __restrict__ deg,
                                            const int32_t* state, bool& kept_nb, bool& blocked) {
  const int gl = threadIdx.x & (GW - 1);
  const int wd0 = b0 + gl;
  uint64_t wv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) wv[u] = wd0 + GW * u < W ? row[wd0 + GW * u] : 0ull;
#pragma unroll
  for (int u = 0; u < U; ++u) {
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
}

// A kept position q offers itself to every neighbour, as soon as it is
// kept: it marks the neighbour absorbed (a neighbour of a kept position is
// never kept, so it ends absorbed) and keeps in claim[b] the largest key
// (degree << 32 | ~position), i.e. the neighbour's first kept neighbour in
// walk order.  The maximum does not depend on when each kept position makes
// its claims, so every pass that keeps a position claims for it at once and
// no pass over the kept rows is needed afterwards.  The GW lanes of q's group
// share the row, four words a lane at a time.
template <int GW>
__device__ __forceinline__ void greedy_claim(int q, int dq, int lo, int n, int W,
                                             const uint64_t* __restrict__ row, int32_t* state,
                                             unsigned long long* __restrict__ claim) {
  const int gl = threadIdx.x & (GW - 1);
  const unsigned long long key = (static_cast<unsigned long long>(dq) << 32) |
                                 static_cast<unsigned int>(~static_cast<unsigned int>(q));
  constexpr int U = 4;
  for (int wd0 = gl; wd0 < W; wd0 += U * GW) {
    uint64_t wv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) wv[u] = wd0 + GW * u < W ? row[wd0 + GW * u] : 0ull;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t bits = wv[u];
      const int cbase = (wd0 + GW * u) * 64;
      while (bits) {
        const int b = __ffsll(static_cast<long long>(bits)) - 1;
        bits &= bits - 1;
        if (cbase + b < n) {
          store_flag(&state[lo + cbase + b], kStateAbsorbed);
          atomicMax(&claim[lo + cbase + b], key);
        }
      }
    }
  }
}

// Visit of undecided position p by a GW-lane group: kept if no neighbour is
// kept or undecided with higher priority (it then claims its neighbours at
// once), absorbed if a neighbour is kept, else left undecided (returns
// true).  The row is scanned in chunks and the
// group stops at its first kept or blocking neighbour: the first chunk has
// 4 words a lane (most rows stop there), later ones 8, so that a row
// scanned to its end (every neighbour of lower priority) takes half the
// dependent round trips.
template <bool FRESH, int GW>
__device__ __forceinline__ bool greedy_visit(int p, int lo, int n, int W,
                                             const uint64_t* __restrict__ row,
                                             const int32_t* __restrict__ deg, int32_t* state,
                                             unsigned long long* __restrict__ claim) {
  const int lane = threadIdx.x & 63;
  const int gl = lane & (GW - 1);
  const int gshift = lane & ~(GW - 1);
  const uint64_t gmask = GW == 64 ? ~0ull : ((1ull << (GW & 63)) - 1);
  const int dp = deg[p];
  bool kept_nb = false, blocked = false;
  greedy_scan<FRESH, GW, 4>(0, p, dp, lo, n, W, row, deg, state, kept_nb, blocked);
  for (int b0 = 4 * GW; b0 < W && !((__ballot(kept_nb || blocked) >> gshift) & gmask); b0 += 8 * GW)
    greedy_scan<FRESH, GW, 8>(b0, p, dp, lo, n, W, row, deg, state, kept_nb, blocked);
  const bool any_kept = ((__ballot(kept_nb) >> gshift) & gmask) != 0;
  const bool any_blocked = ((__ballot(blocked) >> gshift) & gmask) != 0;
  if (any_kept) {
    if (gl == 0) store_flag(&state[p], kStateAbsorbed);
    return false;
  }
  if (!any_blocked) {
    if (gl == 0) store_flag(&state[p], kStateKept);
    greedy_claim<GW>(p, dp, lo, n, W, row, state, claim);
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

// The first round over all positions (16 lanes each); also publishes the
// degrees.  On a union of cliques it decides every position: the first
// member of each clique in walk order is kept and claims the others.
__global__ __launch_bounds__(256) void greedy_round_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state, unsigned long long* __restrict__ claim,
    int32_t* __restrict__ degree_out) {
  __shared__ int soff[kMaxExperts + 1];
  if (*err) return;
  load_offsets(offsets, E, soff);
  const int p = blockIdx.x * kVisitPerBlock + (threadIdx.x / kVisitLanes);
  const int gl = threadIdx.x & (kVisitLanes - 1);
  if (p >= soff[E]) return;
  if (degree_out && gl == 0) degree_out[p] = deg[p];
  // every state starts undecided and is written in this round only by p's
  // own visit or as absorbed by a kept neighbour's claims; p's visit can
  // then only find it absorbed again or leave it, so it is not read
  const int e = bucket_of(soff, E, p);
  const int lo = soff[e], n = soff[e + 1] - lo, W = (n + 63) / 64;
  greedy_visit<false, kVisitLanes>(p, lo, n, W, bitmask + bm_off[e] + static_cast<long long>(p - lo) * W, deg,
                                   state, claim);
}

// The round after the grid rounds: a persistent grid, 16 lanes per
// position, that passes over every position (each group reads the states of
// 16 consecutive positions with one load; decided ones cost nothing more)
// and revisits a blocked one a bounded number of times, reading
// the states coherently, so a dependency chain of length L resolves in
// about L visits inside one launch instead of L launches (graphs whose
// chains the grid rounds leave unfinished).  left[0] records that a
// position is still undecided after it, for the finishing pass.
__global__ __launch_bounds__(256) void greedy_more_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state, unsigned long long* __restrict__ claim,
    int* __restrict__ left) {
  __shared__ int soff[kMaxExperts + 1];
  if (*err) return;
  load_offsets(offsets, E, soff);
  const int gl = threadIdx.x & (kVisitLanes - 1);
  const int gshift = threadIdx.x & 63 & ~(kVisitLanes - 1);
  const int S = soff[E];
  // a group reads the states of kVisitLanes consecutive positions with one
  // load and visits the undecided ones among them (most are decided by now)
  for (int base = (blockIdx.x * kVisitPerBlock + static_cast<int>(threadIdx.x) / kVisitLanes) * kVisitLanes;
       base < S; base += gridDim.x * kVisitPerBlock * kVisitLanes) {
    const int pq = base + gl;
    const bool und = pq < S && load_flag(&state[pq]) == kStateUndecided;
    uint32_t m = static_cast<uint32_t>((__ballot(und) >> gshift) & ((1ull << kVisitLanes) - 1));
    while (m) {
      const int p = base + __ffs(m) - 1;
      m &= m - 1;
      const int e = bucket_of(soff, E, p);
      const int lo = soff[e], n = soff[e + 1] - lo, W = (n + 63) / 64;
      const uint64_t* row = bitmask + bm_off[e] + static_cast<long long>(p - lo) * W;
      bool still = greedy_visit<true, kVisitLanes>(p, lo, n, W, row, deg, state, claim);
      for (int pass = 1; still && pass < kGreedyPasses; ++pass) {
        __builtin_amdgcn_s_sleep(32);
        still = greedy_visit<true, kVisitLanes>(p, lo, n, W, row, deg, state, claim);
      }
      if (still && gl == 0) store_flag(&left[0], 1);
    }
  }
}

// One workgroup per bucket decides what the grid rounds left.  The
// undecided positions are gathered into a list in LDS (a coalesced pass over
// the bucket's states); at most kFinishRounds rounds then visit only the
// listed positions, 16 lanes each (64 at a time), keeping those still
// undecided for the next round (a round decides at least the
// highest-priority undecided position; on clustered data one or two rounds
// decide all).  What is left after them (dependency chains, such as a path
// of similar tokens) is sorted by priority (degree descending, position
// ascending; a bitonic sort in LDS) and visited once each in that order by
// one wave: every higher-priority neighbour of a position is decided by its
// turn, so each visit decides its position, and the work is bounded by one
// visit per position instead of one per position and round.  A bucket with
// more undecided positions than the list holds first runs rounds over all
// its positions until the rest fits the list.
constexpr int kFinishList = 16384;
constexpr int kFinishRounds = 16;

__global__ __launch_bounds__(1024) void greedy_finish_kernel(
    const int32_t* __restrict__ offsets, int E, const long long* __restrict__ bm_off,
    const int* __restrict__ err, const uint64_t* __restrict__ bitmask,
    const int32_t* __restrict__ deg, int32_t* state, unsigned long long* __restrict__ claim,
    const int* __restrict__ left) {
  __shared__ int list[2][kFinishList];
  __shared__ int cnt[2];
  if (*err) return;
  if (load_flag(&left[0]) == 0) return;   // the grid rounds decided every position
  const int e = blockIdx.x;
  const int lo = offsets[e], n = offsets[e + 1] - lo, W = (n + 63) / 64;
  if (n == 0) return;
  const int tid = threadIdx.x;
  const uint64_t* rows = bitmask + bm_off[e];
  int m;
  for (;;) {
    if (tid < 2) cnt[tid] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += 1024) {
      if (load_flag(&state[lo + i]) == kStateUndecided) {
        const int slot = atomicAdd(&cnt[0], 1);
        if (slot < kFinishList) list[0][slot] = i;
      }
    }
    __syncthreads();
    m = cnt[0];
    if (m == 0) return;
    if (m <= kFinishList) break;
    // more than the list holds: a round over all positions, one wave each
    const int wv = tid >> 6;
    for (int pl = wv; pl < n; pl += 16) {
      const int p = lo + pl;
      if (load_flag(&state[p]) != kStateUndecided) continue;
      greedy_visit<true, 64>(p, lo, n, W, rows + static_cast<long long>(pl) * W, deg, state, claim);
    }
    __syncthreads();
  }
  int cur = 0;
  {
    const int grp = tid / kVisitLanes;
    constexpr int kGroups = 1024 / kVisitLanes;
    for (int it = 0; it < kFinishRounds && m > 0; ++it) {
      for (int idx = grp; idx < m; idx += kGroups) {
        const int pl = list[cur][idx];
        greedy_visit<true, kVisitLanes>(lo + pl, lo, n, W, rows + static_cast<long long>(pl) * W, deg, state,
                                        claim);
      }
      if (tid == 0) cnt[cur ^ 1] = 0;
      __syncthreads();
      for (int idx = tid; idx < m; idx += 1024) {
        const int pl = list[cur][idx];
        if (load_flag(&state[lo + pl]) == kStateUndecided) list[cur ^ 1][atomicAdd(&cnt[cur ^ 1], 1)] = pl;
      }
      __syncthreads();
      cur ^= 1;
      m = cnt[cur];
      __syncthreads();
    }
  }
  if (m == 0) return;
  // sort the m positions left by priority: list[cur] positions, list[cur ^ 1]
  // their degrees; padded to a power of two with entries after every real one
  int* pos = list[cur];
  int* dg = list[cur ^ 1];
  int P = 1;
  while (P < m) P <<= 1;
  for (int i = tid; i < P; i += 1024) {
    if (i < m) dg[i] = deg[lo + pos[i]];
    else { pos[i] = 0x7fffffff; dg[i] = -1; }
  }
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += 1024) {
        const int l = i ^ j;
        if (l > i) {
          // a_first: entry i comes before entry l (higher degree, then lower position)
          const bool a_first = dg[i] > dg[l] || (dg[i] == dg[l] && pos[i] < pos[l]);
          const bool up = (i & k) == 0;
          if (up != a_first) {
            const int tp = pos[i], td = dg[i];
            pos[i] = pos[l];
            dg[i] = dg[l];
            pos[l] = tp;
            dg[l] = td;
          }
        }
      }
      __syncthreads();
    }
  }
  if (tid < 64) {
    for (int idx = 0; idx < m; ++idx) {
      const int pl = pos[idx];
      greedy_visit<true, 64>(lo + pl, lo, n, W, rows + static_cast<long long>(pl) * W, deg, state, claim);
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
  // history calls only: the previous block's classes in this block's
  // layout, and the pair / tile counters when the caller passes none
  uint64_t* rb_hi = nullptr;
  uint64_t* rb_lo = nullptr;
  unsigned long long* stats = nullptr;
  int* left;                    // a position stayed undecided after the greedy rounds
  int32_t* colinfo = nullptr;   // previous positions of every slot of every position
  int* queue = nullptr;         // tile queues of the similarity kernel
  // the fp8 screen (calls without history whose shape allows it): fp8 rows
  // (and a zero row), their quantisation errors, the tiles left to the bf16
  // pass and their count
  uint8_t* x8 = nullptr;
  float* rho = nullptr;
  int* list = nullptr;
  int* list_count = nullptr;
};

// Process-wide switch of the fp8 similarity screen (on by default).
std::atomic<int> g_gram_screen{1};

// Shapes whose similarity call may take the fp8 screen: long products
// (d >= 2048, whole 128-value fp8 stages) and buckets of MFMA-bound size
// on average (T k / E >= 512); below that the extra pass over x costs
// about what the screen saves.
bool gram_screen_shape(int T, int d, int E, int k) {
  return d >= 2048 && d % 128 == 0 && static_cast<long long>(T) * k >= 512ll * E;
}

// Upper bound of the number of similarity tiles: sum over buckets of
// t_e (t_e + 1) / 2 with t_e = ceil(n_e / kTile) <= ceil(max_bucket / kTile)
// and sum t_e <= S / kTile + E.
long long gram_tile_bound(long long S, int E, int max_bucket) {
  const long long tmax = (static_cast<long long>(max_bucket) + kTile - 1) / kTile;
  return (S / kTile + E) * (tmax + 1) / 2 + 1;
}

CondenseWs carve_condense(Carver& c, int T, int d, int E, int k, int max_bucket, bool history = false) {
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
  w.left = c.take<int>(1);
  w.cap_words = S * ((static_cast<long long>(max_bucket) + 63) / 64);
  w.bitmask = c.take<uint64_t>(static_cast<size_t>(w.cap_words));
  if (history) {
    w.rb_hi = c.take<uint64_t>(static_cast<size_t>(w.cap_words));
    w.rb_lo = c.take<uint64_t>(static_cast<size_t>(w.cap_words));
    w.stats = c.take<unsigned long long>(4);
    w.colinfo = c.take<int32_t>(static_cast<size_t>(S) * k);
    w.queue = c.take<int>(kTileQueues);
  } else if (gram_screen_shape(T, d, E, k)) {
    w.x8 = c.take<uint8_t>(static_cast<size_t>(T + 1) * d);
    w.rho = c.take<float>(T);
    w.list_count = c.take<int>(1);
    w.list = c.take<int>(static_cast<size_t>(gram_tile_bound(S, E, max_bucket)));
  }
  return w;
}

// Arguments of a call with historical similarity.
struct HistCall {
  const int32_t* slot_pos;   // this block's slot positions (for its record)
  const void* in;            // previous block's record or nullptr
  void* out;                 // this block's record or nullptr
  float S1, S2;
  unsigned long long* stats;
};

}  // namespace
}  // namespace luffy

using namespace luffy;

namespace {

int condense_check(const char* fn, const void* x, int T, int d, int dtype, const int32_t* perm_token,
                   const int32_t* offsets, int E, int k, int max_bucket, float threshold, const int32_t* rep_of_pos,
                   const int32_t* rep_row, const int32_t* rep_offsets, const int32_t* rep_token) {
  if (!x || !perm_token || !offsets || !rep_of_pos || !rep_row || !rep_offsets || !rep_token)
    return fail(LUFFY_E_INVALID, "%s: null pointer argument", fn);
  if (T <= 0 || d <= 0 || E <= 0 || max_bucket < 0)
    return fail(LUFFY_E_INVALID, "%s: T=%d d=%d E=%d max_bucket=%d", fn, T, d, E, max_bucket);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "%s: k=%d must be 1 or 2", fn, k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16) return fail(LUFFY_E_INVALID, "%s: unknown dtype %d", fn, dtype);
  if (threshold != threshold) return fail(LUFFY_E_INVALID, "%s: threshold is NaN", fn);
  if (E > kMaxExperts) return fail(LUFFY_E_UNSUPPORTED, "%s: E=%d > %d", fn, E, kMaxExperts);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "%s: d=%d not a multiple of 64", fn, d);
  if (d > 32768) return fail(LUFFY_E_UNSUPPORTED, "%s: d=%d > 32768", fn, d);
  if (static_cast<long long>(T) * d * elem_bytes(dtype) > 0xFFFF0000ll)
    return fail(LUFFY_E_UNSUPPORTED, "%s: x exceeds 4 GiB - 64 KiB", fn);
  if (static_cast<long long>(T) * k > (1ll << 24)) return fail(LUFFY_E_UNSUPPORTED, "%s: T*k > 2^24", fn);
  return LUFFY_OK;
}

// Every launch of a condense call; hc is null for a call without history.
void condense_enqueue(const void* x, int T, int d, int dtype, const int32_t* perm_token, const int32_t* offsets,
                      int E, int k, int max_bucket, float threshold, int32_t* rep_of_pos, int32_t* rep_row,
                      int32_t* rep_offsets, int32_t* rep_token, void* x_rep, int32_t* degree,
                      const float* inv_norm, const CondenseWs& ws, const HistCall* hc, hipStream_t s) {
  const int S = T * k;
  const bool bf16 = dtype == LUFFY_BF16;
  unsigned long long* stats = hc ? (hc->stats ? hc->stats : ws.stats) : nullptr;
  // norms from the caller when given (the gate pass already read x)
  const float* inv_norm_use = inv_norm ? inv_norm : ws.inv_norm;
  // the fp8 similarity screen: its rows are written by the norm pass
  const bool screen = !hc && bf16 && ws.x8 && threshold > 0.f && g_gram_screen.load(std::memory_order_relaxed);
  const int norm_blocks = screen ? std::max((S + 255) / 256, (T + 4) / 4)
                                 : inv_norm ? std::max(1, (S + 255) / 256) : (T + 3) / 4;
  {
    const int tile = bf16 ? kTile : kTileF32;
#define LUFFY_NORM_ARGS x, T, d, inv_norm ? const_cast<float*>(inv_norm) : ws.inv_norm, S, ws.deg, ws.state, ws.claim, \
                        offsets, E, max_bucket, tile, ws.cap_words, ws.tile_off, ws.bm_off, ws.err, stats, ws.queue,   \
                        ws.left, ws.list_count, ws.x8, ws.rho
    if (bf16 && screen) {
      if (inv_norm) launch("norm", norm_kernel<true, false, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
      else launch("norm", norm_kernel<true, true, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
    } else if (bf16) {
      if (inv_norm) launch("norm", norm_kernel<true, false>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
      else launch("norm", norm_kernel<true, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
    } else {
      if (inv_norm) launch("norm", norm_kernel<false, false>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
      else launch("norm", norm_kernel<false, true>, norm_blocks, 256, 0, s, LUFFY_NORM_ARGS);
    }
#undef LUFFY_NORM_ARGS
  }
  if (!hc) {
    const uint16_t* xb = static_cast<const uint16_t*>(x);
    if (screen) {
      // fp8 screen over every tile, then the bf16 pass over the tiles it left
      launch("gram", gram_kernel_bf16<kGramScreen>, persistent_grid(), GramGemm::THREADS, 0, s,
             reinterpret_cast<const uint16_t*>(ws.x8), d / 2, perm_token, offsets, E, nullptr, threshold,
             ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.rho, ws.list, ws.list_count, T);
      launch("gram_recheck", gram_kernel_bf16<kGramList>, persistent_grid(), GramGemm::THREADS, 0, s, xb, d,
             perm_token, offsets, E, inv_norm_use, threshold, ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg,
             nullptr, ws.list, ws.list_count, T);
    } else if (bf16)
      launch("gram", gram_kernel_bf16<kGramPlain>, persistent_grid(), GramGemm::THREADS, 0, s, xb, d, perm_token,
             offsets, E, inv_norm_use, threshold, ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg, nullptr,
             nullptr, nullptr, T);
    else
      launch("gram", gram_kernel_f32, 2 * persistent_grid(), 256, 0, s, static_cast<const float*>(x), d, perm_token,
             offsets, E, inv_norm_use, threshold, ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg);
  } else {
    Carver cin(const_cast<void*>(hc->in)), cout(hc->out);
    const HistRec rin = carve_hist(cin, T, E, k, max_bucket);
    const HistRec rout = carve_hist(cout, T, E, k, max_bucket);
    if (hc->in) {
      const int blocks = (S + kGatherRows - 1) / kGatherRows + E;
      const int cblocks = std::max(1, std::min(1024, (S + 255) / 256));
      if (k == 1) {
        launch("hist_cols", hist_cols_kernel<1>, cblocks, 256, 0, s, offsets, E, perm_token, ws.err, rin, T,
               max_bucket, ws.colinfo);
        launch("hist_gather", hist_gather_kernel<1>, blocks, 256, 0, s, offsets, E, ws.bm_off, ws.err, rin,
               ws.colinfo, ws.rb_hi, ws.rb_lo);
      } else {
        launch("hist_cols", hist_cols_kernel<2>, cblocks, 256, 0, s, offsets, E, perm_token, ws.err, rin, T,
               max_bucket, ws.colinfo);
        launch("hist_gather", hist_gather_kernel<2>, blocks, 256, 0, s, offsets, E, ws.bm_off, ws.err, rin,
               ws.colinfo, ws.rb_hi, ws.rb_lo);
      }
    }
    if (hc->out)
      launch("hist_header", hist_header_kernel, std::max(1, std::min(1024, (S + 255) / 256)), 256, 0, s,
             hc->slot_pos, T, k, offsets, E, max_bucket, ws.bm_off, ws.err, rout);
    HistParams hp;
    hp.h = threshold;
    hp.S1 = hc->S1;
    hp.S2 = hc->S2;
    hp.out_hi = hc->out ? rout.hi : nullptr;
    hp.out_lo = hc->out ? rout.lo : nullptr;
    hp.rb_hi = hc->in ? ws.rb_hi : nullptr;
    hp.rb_lo = hc->in ? ws.rb_lo : nullptr;
    hp.stats = stats;
    hp.queue = ws.queue;
    const bool hin = hc->in != nullptr, hout = hc->out != nullptr;
#define LUFFY_GH_ARGS d, perm_token, offsets, E, inv_norm_use, hp, ws.tile_off, ws.bm_off, ws.err, ws.bitmask, ws.deg
    if (bf16) {
      const uint16_t* xb = static_cast<const uint16_t*>(x);
      const int g = persistent_grid();
      const int th = GramGemm::THREADS;
      if (hin && hout) launch("gram", gram_hist_kernel_bf16<true, true>, g, th, 0, s, xb, LUFFY_GH_ARGS);
      else if (hin) launch("gram", gram_hist_kernel_bf16<true, false>, g, th, 0, s, xb, LUFFY_GH_ARGS);
      else if (hout) launch("gram", gram_hist_kernel_bf16<false, true>, g, th, 0, s, xb, LUFFY_GH_ARGS);
      else launch("gram", gram_hist_kernel_bf16<false, false>, g, th, 0, s, xb, LUFFY_GH_ARGS);
    } else {
      const float* xf = static_cast<const float*>(x);
      const int g = 2 * persistent_grid();
      if (hin && hout) launch("gram", gram_hist_kernel_f32<true, true>, g, 256, 0, s, xf, LUFFY_GH_ARGS);
      else if (hin) launch("gram", gram_hist_kernel_f32<true, false>, g, 256, 0, s, xf, LUFFY_GH_ARGS);
      else if (hout) launch("gram", gram_hist_kernel_f32<false, true>, g, 256, 0, s, xf, LUFFY_GH_ARGS);
      else launch("gram", gram_hist_kernel_f32<false, false>, g, 256, 0, s, xf, LUFFY_GH_ARGS);
    }
#undef LUFFY_GH_ARGS
  }
  const int wave_blocks = (S + 3) / 4;
  const int visit_blocks = (S + kVisitPerBlock - 1) / kVisitPerBlock;
  launch("greedy_round", greedy_round_kernel, visit_blocks, 256, 0, s, offsets, E, ws.bm_off, ws.err, ws.bitmask,
         ws.deg, ws.state, ws.claim, degree);
  launch("greedy_more", greedy_more_kernel, std::min(visit_blocks, persistent_grid()), 256, 0, s, offsets, E,
         ws.bm_off, ws.err, ws.bitmask, ws.deg, ws.state, ws.claim, ws.left);
  launch("greedy_finish", greedy_finish_kernel, E, 1024, 0, s, offsets, E, ws.bm_off, ws.err, ws.bitmask, ws.deg,
         ws.state, ws.claim, ws.left);
  const int pos_blocks = (S + 1023) / 1024;
  launch("rep_local", rep_local_kernel, pos_blocks, 1024, 0, s, offsets, E, ws.err, ws.state, ws.claim, rep_of_pos,
         ws.local, ws.bsum, S);
  launch("rep_finalize", rep_finalize_kernel, pos_blocks, 1024, (pos_blocks + 1) * sizeof(int), s, offsets, E,
         rep_of_pos, perm_token, ws.local, ws.bsum, rep_row, rep_token, rep_offsets, S);
  if (x_rep) {
    launch("gather", gather_kernel, wave_blocks, 256, 0, s, static_cast<const uint8_t*>(x),
           static_cast<size_t>(d) * elem_bytes(dtype), rep_offsets, E, rep_token, static_cast<uint8_t*>(x_rep));
  }
}

}  // namespace

extern "C" size_t luffy_condense_workspace_size(int T, int d, int E, int k, int max_bucket) {
  if (T <= 0 || E <= 0 || k <= 0 || max_bucket < 0) return 0;
  Carver c(nullptr);
  carve_condense(c, T, d, E, k, max_bucket);
  return c.size();
}

extern "C" int luffy_condense(const void* x, int T, int d, int dtype,
                              const int32_t* perm_token, const int32_t* offsets,
                              int E, int k, int max_bucket, float threshold,
                              int32_t* rep_of_pos, int32_t* rep_row,
                              int32_t* rep_offsets, int32_t* rep_token,
                              void* x_rep, int32_t* degree, const float* inv_norm,
                              void* workspace, size_t workspace_bytes, void* stream) {
  const int st = condense_check("luffy_condense", x, T, d, dtype, perm_token, offsets, E, k, max_bucket, threshold,
                                rep_of_pos, rep_row, rep_offsets, rep_token);
  if (st != LUFFY_OK) return st;
  const size_t need = luffy_condense_workspace_size(T, d, E, k, max_bucket);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_condense: workspace needs %zu bytes, 256-aligned", need);
  Carver c(workspace);
  const CondenseWs ws = carve_condense(c, T, d, E, k, max_bucket);
  condense_enqueue(x, T, d, dtype, perm_token, offsets, E, k, max_bucket, threshold, rep_of_pos, rep_row,
                   rep_offsets, rep_token, x_rep, degree, inv_norm, ws, nullptr, static_cast<hipStream_t>(stream));
  return check_launch("luffy_condense");
}

extern "C" int luffy_set_similarity_screen(int on) { return g_gram_screen.exchange(on ? 1 : 0); }

extern "C" int luffy_similarity_screen_applies(int T, int d, int E, int k, int dtype) {
  return dtype == LUFFY_BF16 && T > 0 && E > 0 && k > 0 && gram_screen_shape(T, d, E, k) &&
         g_gram_screen.load(std::memory_order_relaxed);
}

extern "C" size_t luffy_history_size(int T, int E, int k, int max_bucket) {
  if (T <= 0 || E <= 0 || k <= 0 || max_bucket < 0) return 0;
  Carver c(nullptr);
  carve_hist(c, T, E, k, max_bucket);
  return c.size();
}

extern "C" size_t luffy_condense_history_workspace_size(int T, int d, int E, int k, int max_bucket) {
  if (T <= 0 || E <= 0 || k <= 0 || max_bucket < 0) return 0;
  Carver c(nullptr);
  carve_condense(c, T, d, E, k, max_bucket, true);
  return c.size();
}

extern "C" int luffy_condense_history(const void* x, int T, int d, int dtype,
                                      const int32_t* perm_token, const int32_t* offsets,
                                      const int32_t* slot_pos, int E, int k, int max_bucket,
                                      float threshold, const void* hist_in, void* hist_out,
                                      float S1, float S2,
                                      int32_t* rep_of_pos, int32_t* rep_row,
                                      int32_t* rep_offsets, int32_t* rep_token,
                                      void* x_rep, int32_t* degree, const float* inv_norm,
                                      unsigned long long* stats,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "luffy_condense_history";
  const int st = condense_check(fn, x, T, d, dtype, perm_token, offsets, E, k, max_bucket, threshold, rep_of_pos,
                                rep_row, rep_offsets, rep_token);
  if (st != LUFFY_OK) return st;
  if (hist_out && !slot_pos) return fail(LUFFY_E_INVALID, "%s: hist_out needs slot_pos", fn);
  if (S1 != S1 || S2 != S2) return fail(LUFFY_E_INVALID, "%s: S1 or S2 is NaN", fn);
  if (hist_in && hist_in == hist_out) return fail(LUFFY_E_INVALID, "%s: hist_in and hist_out alias", fn);
  if ((reinterpret_cast<uintptr_t>(hist_in) & 255u) || (reinterpret_cast<uintptr_t>(hist_out) & 255u))
    return fail(LUFFY_E_INVALID, "%s: records must be 256-byte aligned", fn);
  const size_t need = luffy_condense_history_workspace_size(T, d, E, k, max_bucket);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "%s: workspace needs %zu bytes, 256-aligned", fn, need);
  Carver c(workspace);
  const CondenseWs ws = carve_condense(c, T, d, E, k, max_bucket, true);
  HistCall hc{slot_pos, hist_in, hist_out, S1, S2, stats};
  condense_enqueue(x, T, d, dtype, perm_token, offsets, E, k, max_bucket, threshold, rep_of_pos, rep_row,
                   rep_offsets, rep_token, x_rep, degree, inv_norm, ws, &hc, static_cast<hipStream_t>(stream));
  return check_launch(fn);
}
