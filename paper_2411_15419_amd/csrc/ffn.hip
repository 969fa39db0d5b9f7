// luffy_expert_ffn: grouped FFN over the representatives of every expert,
//   H = act(X_rep W1_e^T)   (rounded to the element type)
//   Y = H W2_e^T
// Row counts per expert live on the device: the bf16 kernels are persistent
// (one block per CU) and find their tiles from rep_offsets; the fp32 grid
// is sized from the upper bound ceil(max_rows/64) + E row tiles and blocks
// without a tile exit.
//
// bf16: MFMA tiles of 256 weight rows by 256 or 320 token rows.  The weight
// rows are the P operand and the token rows the Q operand, so each lane
// ends with groups of four consecutive output columns of one row and stores
// each as one 8-byte word.  The last row tile of an expert usually holds
// fewer rows; its waves skip the MFMAs of the missing rows.
// fp32: 64 x 64 tiles of plain FMA (4 x 4 per thread).
#include <type_traits>

#include "gemm_core.h"
#include "luffy_common.h"

namespace luffy {
namespace {

// Activations of the float32 path: exact erf-GELU and SiLU from the device
// math library.
template <int ACT>
__device__ __forceinline__ float act_fn(float z) {
  if constexpr (ACT == LUFFY_ACT_GELU) {
    return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
  } else {
    return z / (1.0f + expf(-z));
  }
}

// Activations of the bf16 path, whose results are rounded to bf16 (relative
// step 2^-8): a dozen VALU operations instead of the library erf, which
// dominated the epilogue of the first product.
//   GELU: erf from Abramowitz & Stegun 7.1.26 (Hastings' rational
//   approximation), erf(u) = 1 - q(u), q(u) = t (a1 + t (a2 + ... + t a5))
//   e^{-u^2}, t = 1 / (1 + p u), u >= 0, |error| <= 1.5e-7.  With
//   u = |z| / sqrt(2): GELU(z) = z (1 - q/2) for z >= 0 and z q/2 for z < 0,
//   evaluated as |z| (1 - q) / 2 + z / 2.
//   SiLU: z / (1 + 2^{-z log2 e}).
// The hardware exp2 and reciprocal are accurate to about 1 ulp.
// Activation code of a plain product (no activation), used by the backward.
constexpr int kActNone = 2;

template <int ACT>
__device__ __forceinline__ float act_fast(float z) {
  if constexpr (ACT == kActNone) {
    return z;
  } else if constexpr (ACT == LUFFY_ACT_GELU) {
    // Hastings' erf(u) = 1 - t (a1 + a2 t + ... + a5 t^4) e^{-u^2},
    // t = 1 / (1 + p u), u = |z| / sqrt(2), with the a_i halved here so
    // that w = 1/2 - t e P(t) = erf(u) / 2.  Then z Phi(z) = |z| w + z / 2
    // for either sign of z (Phi(z) = 1/2 + sign(z) erf(u) / 2): 10 vector
    // operations and two transcendentals per element.
    constexpr float kPs = 0.3275911f * 0.70710678118654752f;   // p / sqrt(2)
    constexpr float kB1 = 0.5f * 0.254829592f, kB2 = 0.5f * -0.284496736f, kB3 = 0.5f * 1.421413741f;
    constexpr float kB4 = 0.5f * -1.453152027f, kB5 = 0.5f * 1.061405429f;
    constexpr float kHalfLog2e = -0.72134752044448170f;   // -log2(e) / 2
    const float a = fabsf(z);
    const float t = __builtin_amdgcn_rcpf(fmaf(kPs, a, 1.0f));
    const float pt = fmaf(t, fmaf(t, fmaf(t, fmaf(t, kB5, kB4), kB3), kB2), kB1);
    const float e = __builtin_amdgcn_exp2f(z * z * kHalfLog2e);   // e^{-u^2}
    const float w = fmaf(-(t * e), pt, 0.5f);
    return fmaf(a, w, 0.5f * z);
  } else {
    constexpr float kNegLog2e = -1.44269504088896341f;
    return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z * kNegLog2e));
  }
}

// Derivative of the activation, with the approximations of act_fast (the
// result is rounded to bf16): GELU'(z) = Phi(z) + z phi(z), Phi from the
// same Hastings erf (Phi(z) = 1 - q/2 for z >= 0, q/2 below), phi(z) =
// e^{-z^2/2} / sqrt(2 pi) from the same exp2; SiLU'(z) = s (1 + z (1 - s)).
template <int ACT>
__device__ __forceinline__ float act_grad(float z) {
  if constexpr (ACT == LUFFY_ACT_GELU) {
    constexpr float kP = 0.3275911f;
    constexpr float kA1 = 0.254829592f, kA2 = -0.284496736f, kA3 = 1.421413741f;
    constexpr float kA4 = -1.453152027f, kA5 = 1.061405429f;
    constexpr float kInvSqrt2 = 0.70710678118654752f, kInvSqrt2Pi = 0.39894228040143268f;
    constexpr float kHalfLog2e = -0.72134752044448170f;   // -log2(e) / 2
    const float u = fabsf(z) * kInvSqrt2;
    const float t = __builtin_amdgcn_rcpf(fmaf(kP, u, 1.0f));
    const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, kA5, kA4), kA3), kA2), kA1);
    const float e = __builtin_amdgcn_exp2f(z * z * kHalfLog2e);   // e^{-z^2/2}
    const float hq = 0.5f * poly * e;
    return (z >= 0.f ? 1.0f - hq : hq) + z * kInvSqrt2Pi * e;
  } else {
    constexpr float kNegLog2e = -1.44269504088896341f;
    const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z * kNegLog2e));
    return sg * (1.0f + z * (1.0f - sg));
  }
}

// Epilogue codes of the backward's dA product: multiply by act'(Z) read
// from a second buffer (dZ = dA * act'(Z)).
constexpr int kActDzGelu = 3, kActDzSilu = 4;

// Row tile q of the ragged row list: expert e, first row row0 and row count.
// Wave-uniform; lane e handles expert e.  Returns false past the last tile.
__device__ __forceinline__ bool locate_row_tile(const int32_t* __restrict__ rep_offsets, int E,
                                                int BM, int q, int& e_out, int& row0, int& rows) {
  const int lane = threadIdx.x & 63;
  int lo = 0, hi = 0, cnt = 0;
  if (lane < E) {
    lo = rep_offsets[lane];
    hi = rep_offsets[lane + 1];
    cnt = (hi - lo + BM - 1) / BM;
  }
  int incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  const uint64_t before = __ballot(lane < E && incl <= q);
  const int e = __popcll(before);
  if (e >= E) return false;
  const int excl = __shfl(incl - cnt, e, 64);
  const int elo = __shfl(lo, e, 64);
  const int ehi = __shfl(hi, e, 64);
  e_out = e;
  row0 = elo + (q - excl) * BM;
  rows = min(BM, ehi - row0);
  return true;
}

// Tile shapes of the bf16 products: 256 output columns (weight rows, the P
// operand) by up to 256 token rows (FfnGemm), or by up to 320 token rows
// (FfnGemmWide).  A tile streams its 256 weight rows once per token tile, so
// an expert whose row count lies in (256, 320] (or (512, 640], ...) needs one
// weight pass fewer with the wide shape; every other expert keeps the
// narrow shape, whose main loop runs a few percent faster (fewer registers,
// smaller stages).  Both shapes share the block size, the LDS buffer and the
// split-K slots.
using FfnGemm = GemmRagged64;
using FfnGemmWide = GemmCore<256, 320, 4, 2, true, false>;
// An expert with at most 128 rows (one token tile of 128) streams its weight
// panels from HBM for little MFMA work, so its tiles are bound by how much
// of the stream one CU has in flight: the 256 x 128 shape takes a ring of
// three 64-wide stages in the same LDS (two in flight while one is
// multiplied, against one for the 256 x 256 shape).
using FfnGemmSmall = GemmCore<256, 128, 4, 2, true, false, 64, 3>;
// The backward's row products read the weights transposed: P K-major.
using FfnGemmT = GemmCore<256, 256, 4, 2, true, false, 64, 2, true, false>;
using FfnGemmWideT = GemmCore<256, 320, 4, 2, true, false, 64, 2, true, false>;
using FfnGemmSmallT = GemmCore<256, 128, 4, 2, true, false, 64, 3, true, false>;
static_assert(FfnGemm::BM == FfnGemmWide::BM && FfnGemm::THREADS == FfnGemmWide::THREADS, "shared tile map");
static_assert(FfnGemm::BM == FfnGemmSmall::BM && FfnGemm::THREADS == FfnGemmSmall::THREADS, "shared tile map");
constexpr int kFfnLds = FfnGemmWide::LDS_BYTES > FfnGemm::LDS_BYTES ? FfnGemmWide::LDS_BYTES : FfnGemm::LDS_BYTES;
static_assert(FfnGemmSmall::LDS_BYTES <= kFfnLds && FfnGemmSmallT::LDS_BYTES <= kFfnLds, "small shape's ring");
// tile shapes of the tile map
constexpr int kShapeNarrow = 0, kShapeWide = 1, kShapeSmall = 2;
// split-K partial tiles: one slot (the accumulators of a tile in register
// layout) per work item, at most kFfnMaxSlots (>= CUs) work items
constexpr int kFfnMaxSlots = 1536;
constexpr size_t kFfnSlotFloats = static_cast<size_t>(FfnGemm::BM) * FfnGemmWide::BN;
// split-K parts cut K at multiples of this (a multiple of both stage widths)
constexpr int kFfnKUnit = 64;
static_assert(kFfnKUnit % FfnGemm::BK == 0 && kFfnKUnit % FfnGemmWide::BK == 0, "K unit");
// Tail counters of the grouped products of one call (forward 2, backward 3).
constexpr int kFfnQueueSets = 3;

// Clears the tail counters of the call's products (a kernel, not a memset,
// so that the call can be captured in a graph).
__global__ __launch_bounds__(64) void ffn_queue_clear_kernel(int* __restrict__ queue, int n) {
  if (static_cast<int>(threadIdx.x) < n) queue[threadIdx.x] = 0;
}

// Tile map of the grouped GEMM (persistent kernels; rep_offsets held one
// expert per lane, E <= 64).  Expert e's rows are cut into tiles of rt_e
// rows (128 for an expert of at most 128 rows, else 256, or 320 where that
// takes fewer tiles); the last one is usually partial.  Tiles are numbered expert by expert; inside an expert,
// output-column tiles come in groups of 4 with the row tiles fastest inside
// a group, so the tiles that share a weight tile run side by side and ~32
// consecutive tiles (one XCD's share of a round, with the XCD-aware block
// numbering) span few weight and token rows.
struct FfnTiles {
  int elo, ehi, rt, mt, incl, NT, tiles;
  __device__ __forceinline__ FfnTiles(const int32_t* __restrict__ rep_offsets, int E, int N) {
    const int lane = threadIdx.x & 63;
    NT = (N + FfnGemm::BM - 1) / FfnGemm::BM;
    elo = ehi = mt = 0;
    rt = FfnGemm::BN;
    if (lane < E) {
      elo = rep_offsets[lane];
      ehi = rep_offsets[lane + 1];
      const int n = ehi - elo;
      constexpr int NB = FfnGemm::BN, WB = FfnGemmWide::BN, SB = FfnGemmSmall::BN;
      rt = n <= SB ? SB : ((n + WB - 1) / WB < (n + NB - 1) / NB ? WB : NB);
      mt = (n + rt - 1) / rt;
    }
    incl = mt * NT;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
    tiles = __builtin_amdgcn_readfirstlane(__shfl(incl, 63, 64));
  }
  // Tile t -> expert e, first token row row0, row count, first output n0,
  // and its shape (kShape*).
  __device__ __forceinline__ void decode(int t, int E, int& e, int& row0, int& rows, int& n0, int& shape) const {
    const int lane = threadIdx.x & 63;
    e = __popcll(__ballot(lane < E && incl <= t));
    const int me = __shfl(mt, e, 64);
    const int excl = __shfl(incl, e, 64) - me * NT;
    const int r = t - excl;
    const int ng = (NT + 3) / 4;
    const int g = min(r / (4 * me), ng - 1);
    const int r2 = r - 4 * g * me;
    const int ms = r2 % me, nt = 4 * g + r2 / me;
    // shuffles return vector registers: made scalar again so that the
    // buffer resources built from them stay in scalar registers
    const int rte = __builtin_amdgcn_readfirstlane(__shfl(rt, e, 64));
    row0 = __builtin_amdgcn_readfirstlane(__shfl(elo, e, 64) + ms * rte);
    rows = __builtin_amdgcn_readfirstlane(min(rte, __shfl(ehi, e, 64) - row0));
    n0 = __builtin_amdgcn_readfirstlane(nt * FfnGemm::BM);
    shape = rte == FfnGemmWide::BN ? kShapeWide : (rte == FfnGemmSmall::BN ? kShapeSmall : kShapeNarrow);
  }
  // Split-K parts per tile (second product only).  Only a product with
  // fewer tiles than blocks splits (with more, every CU already has a tile
  // and the partial tiles' round trip costs more than the balance gains:
  // measured on 424 tiles of K = 8192).  It takes the split s in 2..4 (each
  // part at least 4 K-units, every part's partial tile within the slots)
  // with the fewest rounds times part length, ceil(tiles*s/grid)/s in units
  // of a whole tile; ties keep the smaller split.  The per-CU operand
  // stream, not HBM, bounds these products, so rounds of shorter parts on
  // more CUs win even when a round is not full: 140 tiles of K = 4096 take
  // 2 rounds of thirds instead of 2 rounds of halves.
  __device__ __forceinline__ int parts(int grid, int nk) const {
    if (tiles <= 0 || tiles >= grid) return 1;
    int best = 1;
    long long best_cost = 12ll * ((tiles + grid - 1) / grid);
    for (int sp = 2; sp <= 4; ++sp) {
      if (nk / sp < 4 || static_cast<long long>(tiles) * sp > kFfnMaxSlots) break;
      const long long cost = (12 / sp) * ((static_cast<long long>(tiles) * sp + grid - 1) / grid);
      if (cost < best_cost) {
        best_cost = cost;
        best = sp;
      }
    }
    return best;
  }
  // Split plan of the second product: tiles [0, full) run whole, the `tail`
  // tiles after them run as S parts each (items full + u, u < tail * S, are
  // part u % S of tile full + u / S; partial slot u).  With fewer tiles than
  // blocks every tile is a tail tile and S comes from parts().  With more,
  // the whole rounds stay whole and only the tiles left over for the last,
  // partial round are split, into the most parts (at most 4, at least 4
  // K-units each) that one and a half rounds of blocks take: their parts
  // then fill the CUs that finish their whole tiles first instead of
  // leaving them idle (376 tiles of K = 8192 on 256 CUs: the 120 left over
  // in thirds, second product + reduction 358 -> 345 us; halves 350,
  // quarters 346).
  __device__ __forceinline__ void split_plan(int grid, int nk, int& full, int& tail, int& S) const {
    if (tiles < grid) {
      full = 0;
      tail = tiles;
      S = parts(grid, nk);
      return;
    }
    full = tiles / grid * grid;
    tail = tiles - full;
    S = 1;
    for (int sp = 2; sp <= 4; ++sp)
      if (tail > 0 && 2 * tail * sp <= 3 * grid && nk / sp >= 4 && tail * sp <= kFfnMaxSlots) S = sp;
  }
};

// Multiplies with only the first nq of the wave's Q blocks (wave-uniform
// nq in 0..FN), so the MFMAs of token rows past a partial tile are skipped.
template <class G, int N>
__device__ __forceinline__ void run_nq(int nq, const uint16_t* pbase, const uint32_t (&poff)[G::LP],
                                       const uint16_t* qbase, const uint32_t (&qoff)[G::LQ], int K, int pvalid,
                                       int qvalid, uint8_t* lds, typename G::Acc& acc, int pld) {
  if constexpr (N == 0) {
    G::template run<0>(pbase, poff, qbase, qoff, K, pvalid, qvalid, lds, acc, pld);
  } else {
    if (nq >= N) G::template run<N>(pbase, poff, qbase, qoff, K, pvalid, qvalid, lds, acc, pld);
    else run_nq<G, N - 1>(nq, pbase, poff, qbase, qoff, K, pvalid, qvalid, lds, acc, pld);
  }
}

// One output tile (or one K part of it) of shape G: rows row0.. of A
// (through row_index when given) times the weight rows n0.. of We over K
// range [k0, k1).  Stores bf16 (activation applied when FIRST), or, when
// slot is given, the float32 accumulators in register layout: float4 unit
// ((w*FM + fm)*FN + fn)*4 + g of lane l holds acc[fm][fn][4g..4g+3].
template <class G, int ACT, bool FIRST>
__device__ __forceinline__ void ffn_tile(const uint16_t* __restrict__ A, const int32_t* __restrict__ row_index,
                                         const uint16_t* __restrict__ We, int K, int N, int k0, int k1, int row0,
                                         int rows, int n0, uint16_t* __restrict__ out, float* __restrict__ slot,
                                         const uint16_t* __restrict__ aux, uint8_t* lds) {
  static_assert(G::FN <= 5, "ragged dispatch instantiates FN + 1 main loops");
  const int tid = opaque_tid(), lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = G::wave_m(w), wn = G::wave_n(w);
  uint32_t poff[G::LP], qoff[G::LQ];
#pragma unroll
  for (int j = 0; j < G::LP; ++j) {
    // weights [N, K] row-major, or (G::PT) [K, N]: element (k, n) at k * N + n
    if constexpr (G::PT) poff[j] = G::kmajor_offset(j, N, n0, N - n0);
    else poff[j] = static_cast<uint32_t>(min(n0 + G::load_row(j), N - 1)) * K;
  }
#pragma unroll
  for (int j = 0; j < G::LQ; ++j) {
    const int m = row0 + min(G::load_row(G::LP + j) - G::BM, rows - 1);
    qoff[j] = static_cast<uint32_t>(row_index ? row_index[m] : m) * K;
  }
  const int nq = G::active_q(wn, rows);
  typename G::Acc acc;
  G::zero(acc);
  run_nq<G, G::FN>(__builtin_amdgcn_readfirstlane(nq), We + (G::PT ? static_cast<size_t>(k0) * N : k0), poff,
                   A + k0, qoff, k1 - k0, N - n0, rows, lds, acc, N);
  if constexpr (ACT != kActDzGelu && ACT != kActDzSilu) {
    if (!slot) {
      // bf16 rows: lane l (< 32) holds columns 8g..8g+3 and lane l + 32
      // columns 8g+4..8g+7 of a 32-column block of one token row; after one
      // exchange the low lane stores columns 0..15 and the high lane 16..31,
      // two 16-byte stores each
      const int hi = lane >> 5;
#pragma unroll
      for (int fm = 0; fm < G::FM; ++fm) {
#pragma unroll
        for (int fn = 0; fn < G::FN; ++fn) {
          const int ml = G::q_row(wn, fn) + (lane & 31);
          const int nb = n0 + wm * G::WTM + 32 * fm;
          if (ml >= rows || nb >= N) continue;
          uint32_t pk[4][2];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float z[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              z[q] = acc[fm][fn][4 * g + q];
              if constexpr (FIRST) z[q] = act_fast<ACT>(z[q]);
            }
            pk[g][0] = pack_bf16x2(z[0], z[1]);
            pk[g][1] = pack_bf16x2(z[2], z[3]);
          }
          uint32_t snd[4] = {hi ? pk[0][0] : pk[2][0], hi ? pk[0][1] : pk[2][1], hi ? pk[1][0] : pk[3][0],
                             hi ? pk[1][1] : pk[3][1]};
          uint32_t rcv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) rcv[i] = static_cast<uint32_t>(__shfl_xor(static_cast<int>(snd[i]), 32, 64));
          uint4* dst = reinterpret_cast<uint4*>(out + static_cast<size_t>(row0 + ml) * N + nb + 16 * hi);
          if (hi == 0) {
            dst[0] = make_uint4(pk[0][0], pk[0][1], rcv[0], rcv[1]);
            dst[1] = make_uint4(pk[1][0], pk[1][1], rcv[2], rcv[3]);
          } else {
            dst[0] = make_uint4(rcv[0], rcv[1], pk[2][0], pk[2][1]);
            dst[1] = make_uint4(rcv[2], rcv[3], pk[3][0], pk[3][1]);
          }
        }
      }
      return;
    }
  }
#pragma unroll
  for (int fm = 0; fm < G::FM; ++fm) {
#pragma unroll
    for (int fn = 0; fn < G::FN; ++fn) {
      const int ml = G::q_row(wn, fn) + (lane & 31);
      if (ml >= rows) continue;
      uint16_t* orow = out + static_cast<size_t>(row0 + ml) * N;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = wm * G::WTM + 32 * fm + 8 * g + 4 * (lane >> 5);
        const int n = n0 + nl;
        if (n >= N) continue;
        if (slot) {
          // partial tiles keep the accumulator layout: 1 KB per store
          // instruction; the reduction maps it back to rows and columns
          const int u = ((w * G::FM + fm) * G::FN + fn) * 4 + g;
          *reinterpret_cast<float4*>(slot + u * 256 + lane * 4) =
              make_float4(acc[fm][fn][4 * g], acc[fm][fn][4 * g + 1], acc[fm][fn][4 * g + 2],
                          acc[fm][fn][4 * g + 3]);
          continue;
        }
        float z[4];
        if constexpr (ACT == kActDzGelu || ACT == kActDzSilu) {
          // dZ = dA * act'(Z): the four Z values of this store
          const uint2 zw = *reinterpret_cast<const uint2*>(aux + static_cast<size_t>(row0 + ml) * N + n);
          const float zz[4] = {__uint_as_float(zw.x << 16), __uint_as_float(zw.x & 0xFFFF0000u),
                               __uint_as_float(zw.y << 16), __uint_as_float(zw.y & 0xFFFF0000u)};
#pragma unroll
          for (int q = 0; q < 4; ++q)
            z[q] = acc[fm][fn][4 * g + q] * act_grad<ACT == kActDzGelu ? LUFFY_ACT_GELU : LUFFY_ACT_SILU>(zz[q]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            z[q] = acc[fm][fn][4 * g + q];
            if constexpr (FIRST) z[q] = act_fast<ACT>(z[q]);
          }
        }
        *reinterpret_cast<uint2*>(orow + n) = make_uint2(pack_bf16x2(z[0], z[1]), pack_bf16x2(z[2], z[3]));
      }
    }
  }
}

// One product of the FFN for every tile of every expert (persistent).  The
// whole rounds of work items are dealt statically (serpentine, XCD-aware
// block order: consecutive items share weight and token rows in an XCD's
// L2); the items left over, the last ones in the order (the smallest
// experts' tiles), go one at a time through a counter (*tail, zero at
// launch) to the blocks that finish first.  The second product (FIRST =
// false) has few output columns (d); with few representatives it can have
// fewer tiles than CUs, and it then splits K (decided on the device from the
// actual tile count): parts store float32 partial tiles and
// ffn_split_reduce_kernel finishes them.
template <int ACT, bool FIRST, bool WT = false>
__global__ __launch_bounds__(FfnGemm::THREADS) void ffn_kernel_bf16(
    const uint16_t* __restrict__ A, const int32_t* __restrict__ row_index,
    const int32_t* __restrict__ rep_offsets, int E, int K, int N,
    const uint16_t* __restrict__ W, uint16_t* __restrict__ out, float* __restrict__ split_slots,
    const uint16_t* __restrict__ aux, int* __restrict__ tail) {
  // one LDS array: the operand ring, then the block's current tail item (a
  // second LDS variable would cost the K loop its DMA overlap)
  __shared__ __attribute__((aligned(16))) uint8_t lds[kFfnLds + 16];
  int& item_s = *reinterpret_cast<int*>(lds + kFfnLds);
  const FfnTiles map(rep_offsets, E, N);
  const int nk = K / kFfnKUnit;
  int full = map.tiles, ntail = 0, S = 1;
  if (!FIRST) map.split_plan(gridDim.x, nk, full, ntail, S);
  const int total = full + ntail * S;
  // static rounds: whole tiles only when the tail is split (its parts go
  // to the blocks that finish first), else every whole round of items
  const int g = gridDim.x, rounds = (full > 0 && S > 1) ? full / g : total / g;
  const int vb = xcd_virtual_block();
  for (int round = 0;; ++round) {
    int tt;
    if (round < rounds) {
      tt = serpentine_item(round, vb);
    } else {
      if (rounds * g == total) break;   // no tail
      if (threadIdx.x == 0) item_s = rounds * g + atomicAdd(tail, 1);
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the item is in LDS
      raw_barrier();
      // read before the tile's barriers: thread 0 writes the next item only
      // after every thread has passed them
      tt = item_s;
      if (tt >= total) break;
    }
    // whole tile, or part `part` of S of a tail tile (partial slot u)
    const int u = tt - full;
    const int sp = u < 0 ? 1 : S;
    const int t = u < 0 ? tt : full + u / S, part = u < 0 ? 0 : u - (u / S) * S;
    int e, row0, rows, n0, shape;
    map.decode(t, E, e, row0, rows, n0, shape);
    const uint16_t* We = W + static_cast<size_t>(e) * N * K;
    // K range of this part, in whole 64-wide units
    const int k0 = (part * nk / sp) * kFfnKUnit, k1 = ((part + 1) * nk / sp) * kFfnKUnit;
    float* slot = sp > 1 ? split_slots + static_cast<size_t>(u) * kFfnSlotFloats : nullptr;
    using GN = std::conditional_t<WT, FfnGemmT, FfnGemm>;
    using GW = std::conditional_t<WT, FfnGemmWideT, FfnGemmWide>;
    using GS = std::conditional_t<WT, FfnGemmSmallT, FfnGemmSmall>;
    if (shape == kShapeWide)
      ffn_tile<GW, ACT, FIRST>(A, row_index, We, K, N, k0, k1, row0, rows, n0, out, slot, aux, lds);
    else if (shape == kShapeSmall)
      ffn_tile<GS, ACT, FIRST>(A, row_index, We, K, N, k0, k1, row0, rows, n0, out, slot, aux, lds);
    else
      ffn_tile<GN, ACT, FIRST>(A, row_index, We, K, N, k0, k1, row0, rows, n0, out, slot, aux, lds);
  }
}

// Sums the S split parts of unit q (= (w*FM + fm)*FN + fn) of one output
// tile of shape G, lane l, and stores bf16.  The float4 units g = 0..3 of
// lane l hold columns 8g..8g+3 (l < 32) or 8g+4..8g+7 (l >= 32) of a
// 32-column block of one token row; lanes l and l+32 share the row and swap
// halves so that each stores 16 consecutive bf16 (two 16-byte stores).
template <class G, int S>
__device__ __forceinline__ void reduce_unit(const float* __restrict__ slots, int q, int row0, int rows, int n0,
                                            int N, uint16_t* __restrict__ out) {
  const int l = threadIdx.x & 63, hi = l >> 5;
  const int fn = q % G::FN, fm = (q / G::FN) % G::FM, w = q / (G::FN * G::FM);
  const int ml = G::q_row(G::wave_n(w), fn) + (l & 31);
  const int nb = G::wave_m(w) * G::WTM + 32 * fm;   // first column of the 32-column block
  if (ml >= rows || n0 + nb >= N) return;            // same for lanes l and l+32
  const float* src = slots + static_cast<size_t>(q) * 4 * 256 + l * 4;
  // every part's four float4 units loaded before any is added (S is a
  // template constant, so no load waits behind a branch), then summed in
  // part order
  float4 u[S][4];
#pragma unroll
  for (int p = 0; p < S; ++p)
#pragma unroll
    for (int g = 0; g < 4; ++g) u[p][g] = *reinterpret_cast<const float4*>(src + p * kFfnSlotFloats + g * 256);
  float4 v[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    v[g] = u[0][g];
#pragma unroll
    for (int p = 1; p < S; ++p) {
      v[g].x += u[p][g].x; v[g].y += u[p][g].y; v[g].z += u[p][g].z; v[g].w += u[p][g].w;
    }
  }
  // lane l (< 32) holds columns 8g..8g+3, lane l+32 columns 8g+4..8g+7:
  // the low lane keeps columns 0..15, the high lane 16..31
  float4 send[2] = {hi ? v[0] : v[2], hi ? v[1] : v[3]};
  float4 recv[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    recv[i].x = __shfl_xor(send[i].x, 32, 64);
    recv[i].y = __shfl_xor(send[i].y, 32, 64);
    recv[i].z = __shfl_xor(send[i].z, 32, 64);
    recv[i].w = __shfl_xor(send[i].w, 32, 64);
  }
  const float4 c[4] = {hi ? recv[0] : v[0], hi ? v[2] : recv[0], hi ? recv[1] : v[1], hi ? v[3] : recv[1]};
  uint4* dst = reinterpret_cast<uint4*>(out + static_cast<size_t>(row0 + ml) * N + n0 + nb + 16 * hi);
  dst[0] = make_uint4(pack_bf16x2(c[0].x, c[0].y), pack_bf16x2(c[0].z, c[0].w), pack_bf16x2(c[1].x, c[1].y),
                      pack_bf16x2(c[1].z, c[1].w));
  dst[1] = make_uint4(pack_bf16x2(c[2].x, c[2].y), pack_bf16x2(c[2].z, c[2].w), pack_bf16x2(c[3].x, c[3].y),
                      pack_bf16x2(c[3].z, c[3].w));
}

// Sums the split parts of every split (tail) tile in part order and stores
// bf16.  Recomputes the same tile map and split plan, so it does nothing
// when the product was not split.  One thread per (w, fm, fn, lane) unit of a tile;
// a tile gets the block count of the wide shape (the narrow shape leaves
// its last blocks idle).
constexpr int kReduceUnits = FfnGemmWide::NWAVES * FfnGemmWide::FM * FfnGemmWide::FN * 64;
static_assert(kReduceUnits % 256 == 0 &&
                  FfnGemm::NWAVES * FfnGemm::FM * FfnGemm::FN * 64 <= kReduceUnits, "reduction blocks");

__global__ __launch_bounds__(256) void ffn_split_reduce_kernel(const int32_t* __restrict__ rep_offsets, int E,
                                                               int K, int N, const float* __restrict__ split_slots,
                                                               uint16_t* __restrict__ out, int grid_parts) {
  constexpr int PER_TILE = kReduceUnits / 256;   // blocks per tile
  const FfnTiles map(rep_offsets, E, N);
  int full, ntail, S;
  map.split_plan(grid_parts, K / kFfnKUnit, full, ntail, S);
  if (S == 1) return;
  for (int b = blockIdx.x; b < ntail * PER_TILE; b += gridDim.x) {
    const int tt = b / PER_TILE;                                    // tail tile
    const int q = ((b - tt * PER_TILE) * 256 + threadIdx.x) >> 6;   // (w*FM + fm)*FN + fn
    int e, row0, rows, n0, shape;
    map.decode(full + tt, E, e, row0, rows, n0, shape);
    const float* slots = split_slots + static_cast<size_t>(tt) * S * kFfnSlotFloats;
    const bool narrow_unit = q < FfnGemm::NWAVES * FfnGemm::FM * FfnGemm::FN;
    const bool small_unit = q < FfnGemmSmall::NWAVES * FfnGemmSmall::FM * FfnGemmSmall::FN;
    if (S == 4) {
      if (shape == kShapeWide) reduce_unit<FfnGemmWide, 4>(slots, q, row0, rows, n0, N, out);
      else if (shape == kShapeSmall) { if (small_unit) reduce_unit<FfnGemmSmall, 4>(slots, q, row0, rows, n0, N, out); }
      else if (narrow_unit) reduce_unit<FfnGemm, 4>(slots, q, row0, rows, n0, N, out);
    } else if (S == 3) {
      if (shape == kShapeWide) reduce_unit<FfnGemmWide, 3>(slots, q, row0, rows, n0, N, out);
      else if (shape == kShapeSmall) { if (small_unit) reduce_unit<FfnGemmSmall, 3>(slots, q, row0, rows, n0, N, out); }
      else if (narrow_unit) reduce_unit<FfnGemm, 3>(slots, q, row0, rows, n0, N, out);
    } else {
      if (shape == kShapeWide) reduce_unit<FfnGemmWide, 2>(slots, q, row0, rows, n0, N, out);
      else if (shape == kShapeSmall) { if (small_unit) reduce_unit<FfnGemmSmall, 2>(slots, q, row0, rows, n0, N, out); }
      else if (narrow_unit) reduce_unit<FfnGemm, 2>(slots, q, row0, rows, n0, N, out);
    }
  }
}

constexpr int kF32Tile = 64;

// float32 products: 64 x 64 tiles, 4 x 4 outputs per thread, K in chunks of
// 32 through LDS.  Each thread stages 8 elements of each operand per chunk;
// its rows are fixed for the tile (looked up once), and the next chunk's
// elements are loaded into registers while the current one is multiplied.
template <int ACT, bool FIRST>
__global__ __launch_bounds__(256) void ffn_kernel_f32(
    const float* __restrict__ A, const int32_t* __restrict__ row_index,
    const int32_t* __restrict__ rep_offsets, int E, int K, int N,
    const float* __restrict__ W, float* __restrict__ out) {
  constexpr int KC = 32;
  constexpr int PER = kF32Tile * KC / 256;   // staged elements per thread and operand
  __shared__ float As[kF32Tile][KC + 1];
  __shared__ float Bs[kF32Tile][KC + 1];
  int e, row0, rows;
  if (!locate_row_tile(rep_offsets, E, kF32Tile, blockIdx.x, e, row0, rows)) return;
  const int tid = threadIdx.x;
  const int n0 = blockIdx.y * kF32Tile;
  const float* We = W + static_cast<size_t>(e) * N * K;
  const int rb = (tid >> 4) * 4, cb = (tid & 15) * 4;
  // staged element i of this thread: row r0 + 8i (r0 = tid / 32), column kk
  const int kk = tid % KC, r0 = tid / KC;
  const float* ap[PER];
  const float* bp[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int r = r0 + 8 * i;
    const int m = row0 + min(r, rows - 1);
    ap[i] = A + static_cast<size_t>(row_index ? row_index[m] : m) * K + kk;
    bp[i] = We + static_cast<size_t>(min(n0 + r, N - 1)) * K + kk;
  }
  float va[PER], vb[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    va[i] = ap[i][0];
    vb[i] = bp[i][0];
  }
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += KC) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      As[r0 + 8 * i][kk] = va[i];
      Bs[r0 + 8 * i][kk] = vb[i];
    }
    __syncthreads();
    if (k0 + KC < K) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        va[i] = ap[i][k0 + KC];
        vb[i] = bp[i][k0 + KC];
      }
    }
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[rb + i][c];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[cb + j][c];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (rb + i >= rows) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + cb + j;
      if (n >= N) continue;
      float z = acc[i][j];
      if constexpr (FIRST) z = act_fn<ACT>(z);
      out[static_cast<size_t>(row0 + rb + i) * N + n] = z;
    }
  }
}

struct FfnWs {
  void* hidden;
  float* split_slots;
  int* queue;   // kFfnQueueSets tail counters
};

FfnWs carve_ffn(Carver& c, int max_rows, int d_ff, int dtype) {
  FfnWs w;
  w.hidden = c.take<uint8_t>(static_cast<size_t>(max_rows) * d_ff * elem_bytes(dtype));
  w.split_slots = nullptr;
  w.queue = nullptr;
  if (dtype == LUFFY_BF16) {
    w.split_slots = c.take<float>(kFfnSlotFloats * kFfnMaxSlots);
    w.queue = c.take<int>(kFfnQueueSets);
  }
  return w;
}


template <int ACT>
void launch_ffn(const void* x, const int32_t* row_index, const int32_t* rep_offsets, int E, int d,
                int d_ff, int dtype, const void* w1, const void* w2, int max_rows, void* y_rep,
                const FfnWs& ws, hipStream_t s) {
  void* hidden = ws.hidden;
  if (dtype == LUFFY_BF16) {
    const int grid = persistent_grid();
    launch("ffn_queue", ffn_queue_clear_kernel, 1, 64, 0, s, ws.queue, 2);
    {
      launch("ffn1", ffn_kernel_bf16<ACT, true>, grid, FfnGemm::THREADS, 0, s, static_cast<const uint16_t*>(x),
             row_index, rep_offsets, E, d, d_ff, static_cast<const uint16_t*>(w1), static_cast<uint16_t*>(hidden),
             ws.split_slots, static_cast<const uint16_t*>(nullptr), ws.queue);
    }
    {
      launch("ffn2", ffn_kernel_bf16<ACT, false>, grid, FfnGemm::THREADS, 0, s,
             static_cast<const uint16_t*>(hidden), nullptr, rep_offsets, E, d_ff, d,
             static_cast<const uint16_t*>(w2), static_cast<uint16_t*>(y_rep), ws.split_slots,
             static_cast<const uint16_t*>(nullptr), ws.queue + 1);
    }
    {
      launch("ffn2_reduce", ffn_split_reduce_kernel, 8 * grid, 256, 0, s, rep_offsets, E, d_ff, d, ws.split_slots,
             static_cast<uint16_t*>(y_rep), grid);
    }
  } else {
    const int mt = (max_rows + kF32Tile - 1) / kF32Tile + E;
    dim3 g1(mt, (d_ff + kF32Tile - 1) / kF32Tile), g2(mt, (d + kF32Tile - 1) / kF32Tile);
    {
      launch("ffn1", ffn_kernel_f32<ACT, true>, g1, 256, 0, s, static_cast<const float*>(x), row_index, rep_offsets,
             E, d, d_ff, static_cast<const float*>(w1), static_cast<float*>(hidden));
    }
    {
      launch("ffn2", ffn_kernel_f32<ACT, false>, g2, 256, 0, s, static_cast<const float*>(hidden), nullptr,
             rep_offsets, E, d_ff, d, static_cast<const float*>(w2), static_cast<float*>(y_rep));
    }
  }
}

// ---------------------------------------------------------------- backward
// Gradients of Y = W2 act(W1 x) on the representatives (bf16):
//   Z = X W1^T (recomputed), dZ = (dY W2) * act'(Z) (in the product's
//   epilogue), dX = dZ W1, dW2 = dY^T act(Z), dW1 = dZ^T X.
// The row products dZ and dX run on the forward's grouped kernel with the
// weights read K-major (no transposed copy: the core's transposing LDS
// reads); the weight gradients contract over an expert's rows, read K-major
// from the row-major activations, with the rows past the expert's read as
// zeros up to the next multiple of 64.

// A = act(Z) over the R = rep_offsets[E] rows of [*, d_ff] (8 per step).
template <int ACT>
__global__ __launch_bounds__(256) void act_rows_kernel(const int32_t* __restrict__ rep_offsets, int E, int d_ff,
                                                       const uint16_t* __restrict__ z, uint16_t* __restrict__ a) {
  const long long n8 = static_cast<long long>(rep_offsets[E]) * d_ff / 8;
  const uint4* zz = reinterpret_cast<const uint4*>(z);
  uint4* aa = reinterpret_cast<uint4*>(a);
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < n8; i += static_cast<long long>(gridDim.x) * 256) {
    const uint4 v = zz[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = pack_bf16x2(act_fast<ACT>(__uint_as_float(w[q] << 16)), act_fast<ACT>(__uint_as_float(w[q] & 0xFFFF0000u)));
    aa[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// xg[r] = x[row_index[r]] for the R rows in use (one wave per row).
__global__ __launch_bounds__(256) void gather_rows_kernel(const int32_t* __restrict__ rep_offsets, int E, int d,
                                                          const uint16_t* __restrict__ x,
                                                          const int32_t* __restrict__ row_index,
                                                          uint16_t* __restrict__ xg) {
  const int R = rep_offsets[E];
  const int lane = threadIdx.x & 63;
  for (int r = blockIdx.x * 4 + (threadIdx.x >> 6); r < R; r += gridDim.x * 4) {
    const uint4* src = reinterpret_cast<const uint4*>(x + static_cast<size_t>(row_index[r]) * d);
    uint4* dst = reinterpret_cast<uint4*>(xg + static_cast<size_t>(r) * d);
    for (int c = lane; c < d / 8; c += 64) dst[c] = src[c];
  }
}

// First row and K extent (R_e rounded up to 64) of expert e.
__device__ __forceinline__ void expert_rows(const int32_t* __restrict__ rep_offsets, int e, int& lo, int& re) {
  lo = rep_offsets[e];
  re = rep_offsets[e + 1] - lo;
}

// Weight gradients: out[e][i][j] = sum over the expert's rows r of
// P[r][i] Q[r][j], P [*, M] and Q [*, N] row-major token rows (both read
// K-major: the contraction runs over rows); float32 output [E][M][N]; an
// expert without rows gets zeros.
using WgradGemm = GemmCore<256, 256, 2, 4, false, false, 64, 2, true, true>;

// OUT_BF16: the sums are rounded to bf16 (the weights' own type), stored
// four bytes at a time: lanes l and l^1 hold neighbouring columns of the
// same rows and swap one value, so that the even lane stores its row v and
// the odd lane row v+1, two columns each.
template <bool OUT_BF16>
__global__ __launch_bounds__(WgradGemm::THREADS) void wgrad_kernel(const uint16_t* __restrict__ P,
                                                                   const uint16_t* __restrict__ Q,
                                                                   const int32_t* __restrict__ rep_offsets, int E,
                                                                   int M, int N, void* __restrict__ out) {
  using G = WgradGemm;
  __shared__ __attribute__((aligned(16))) uint8_t lds[G::LDS_BYTES];
  const int mt = (M + G::BM - 1) / G::BM, nt = (N + G::BN - 1) / G::BN;
  const int tpe = mt * nt;
  for (int t = blockIdx.x; t < E * tpe; t += gridDim.x) {
    const int e = t / tpe, r = t - e * tpe;
    const int m0 = (r / nt) * G::BM, n0 = (r % nt) * G::BN;
    int lo, re;
    expert_rows(rep_offsets, e, lo, re);
    lo = __builtin_amdgcn_readfirstlane(lo);
    re = __builtin_amdgcn_readfirstlane(re);
    typename G::Acc acc;
    G::zero(acc);
    if (re > 0) {
      uint32_t poff[G::LP], qoff[G::LQ];
#pragma unroll
      for (int j = 0; j < G::LP; ++j) poff[j] = G::kmajor_offset(j, M, m0, M - m0);
#pragma unroll
      for (int j = 0; j < G::LQ; ++j) qoff[j] = G::kmajor_offset(G::LP + j, N, n0, N - n0);
      G::template run<G::FN>(P + static_cast<size_t>(lo) * M, poff, Q + static_cast<size_t>(lo) * N, qoff,
                             (re + 63) / 64 * 64, M - m0, N - n0, lds, acc, M, N, re);
    }
    const int tid = opaque_tid(), lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = G::wave_m(w), wn = G::wave_n(w);
    if constexpr (OUT_BF16) {
      uint16_t* oe = static_cast<uint16_t*>(out) + static_cast<size_t>(e) * M * N;
      const bool odd = lane & 1;
#pragma unroll
      for (int fm = 0; fm < G::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < G::FN; ++fn) {
          // first column of the lane pair; N is a multiple of 64, so both
          // columns are in range or neither is (same for both lanes)
          const int jp = (n0 + G::q_row(wn, fn) + (lane & 31)) & ~1;
          if (jp >= N) continue;
#pragma unroll
          for (int v = 0; v < 16; v += 2) {
            // the even lane needs the odd lane's row-v value, the odd lane
            // the even lane's row-(v+1) value
            const float recv = __shfl_xor(odd ? acc[fm][fn][v] : acc[fm][fn][v + 1], 1, 64);
            const float lo = odd ? recv : acc[fm][fn][v];
            const float hi = odd ? acc[fm][fn][v + 1] : recv;
            const int i = m0 + wm * G::WTM + 32 * fm + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4) + (odd ? 1 : 0);
            if (i < M)
              *reinterpret_cast<uint32_t*>(oe + static_cast<size_t>(i) * N + jp) = pack_bf16x2(lo, hi);
          }
        }
    } else {
      float* oe = static_cast<float*>(out) + static_cast<size_t>(e) * M * N;
#pragma unroll
      for (int fm = 0; fm < G::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < G::FN; ++fn) {
          const int j = n0 + G::q_row(wn, fn) + (lane & 31);
          if (j >= N) continue;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int i = m0 + wm * G::WTM + 32 * fm + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
            if (i < M) oe[static_cast<size_t>(i) * N + j] = acc[fm][fn][v];
          }
        }
    }
  }
}

struct FfnBwdWs {
  uint16_t *z, *a, *dz, *xg;
  float* split_slots;
  int* queue;   // kFfnQueueSets tail counters
};

FfnBwdWs carve_ffn_bwd(Carver& c, int max_rows, int E, int d, int d_ff) {
  (void)E;
  FfnBwdWs w;
  w.z = c.take<uint16_t>(static_cast<size_t>(max_rows) * d_ff);
  w.a = c.take<uint16_t>(static_cast<size_t>(max_rows) * d_ff);
  w.dz = c.take<uint16_t>(static_cast<size_t>(max_rows) * d_ff);
  w.xg = c.take<uint16_t>(static_cast<size_t>(max_rows) * d);
  w.split_slots = c.take<float>(kFfnSlotFloats * kFfnMaxSlots);
  w.queue = c.take<int>(kFfnQueueSets);
  return w;
}

template <int ACT>
void launch_ffn_bwd(const uint16_t* x, const int32_t* row_index, const int32_t* rep_offsets, int E, int d, int d_ff,
                    const uint16_t* w1, const uint16_t* w2, int max_rows, const uint16_t* dy, uint16_t* dx,
                    void* dw1, void* dw2, bool dw_bf16, const FfnBwdWs& ws, hipStream_t s) {
  (void)max_rows;
  const int grid = persistent_grid();
  const int egrid = 4 * grid;
  launch("ffn_queue", ffn_queue_clear_kernel, 1, 64, 0, s, ws.queue, 3);
  // Z = X W1^T, A = act(Z)
  launch("bwd_z", ffn_kernel_bf16<kActNone, true>, grid, FfnGemm::THREADS, 0, s, x, row_index, rep_offsets, E, d,
         d_ff, w1, ws.z, ws.split_slots, static_cast<const uint16_t*>(nullptr), ws.queue);
  launch("bwd_act", act_rows_kernel<ACT>, egrid, 256, 0, s, rep_offsets, E, d_ff, static_cast<const uint16_t*>(ws.z),
         ws.a);
  // dZ = (dY W2) act'(Z): W2 [E][d][d_ff] read K-major (k = output row o)
  constexpr int kDz = ACT == LUFFY_ACT_GELU ? kActDzGelu : kActDzSilu;
  launch("bwd_da", ffn_kernel_bf16<kDz, true, true>, grid, FfnGemm::THREADS, 0, s, dy, nullptr, rep_offsets, E, d,
         d_ff, w2, ws.dz, ws.split_slots, static_cast<const uint16_t*>(ws.z), ws.queue + 1);
  // dX = dZ W1: W1 [E][d_ff][d] read K-major, split over K as the forward's second product
  launch("bwd_dx", ffn_kernel_bf16<kActNone, false, true>, grid, FfnGemm::THREADS, 0, s,
         static_cast<const uint16_t*>(ws.dz), nullptr, rep_offsets, E, d_ff, d, w1, dx, ws.split_slots,
         static_cast<const uint16_t*>(nullptr), ws.queue + 2);
  launch("bwd_dx_reduce", ffn_split_reduce_kernel, 8 * grid, 256, 0, s, rep_offsets, E, d_ff, d, ws.split_slots, dx,
         grid);
  // dW2 = dY^T A, dW1 = dZ^T X (X's rows gathered first)
  auto* wgrad = dw_bf16 ? wgrad_kernel<true> : wgrad_kernel<false>;
  launch("bwd_dw2", wgrad, grid, WgradGemm::THREADS, 0, s, dy, static_cast<const uint16_t*>(ws.a), rep_offsets, E, d,
         d_ff, dw2);
  const uint16_t* xr = x;
  if (row_index) {
    launch("bwd_gather", gather_rows_kernel, egrid, 256, 0, s, rep_offsets, E, d, x, row_index, ws.xg);
    xr = ws.xg;
  }
  launch("bwd_dw1", wgrad, grid, WgradGemm::THREADS, 0, s, static_cast<const uint16_t*>(ws.dz), xr, rep_offsets, E,
         d_ff, d, dw1);
}

}  // namespace
}  // namespace luffy

using namespace luffy;

extern "C" size_t luffy_expert_ffn_workspace_size(int max_rows, int E, int d_ff, int dtype) {
  (void)E;
  if (max_rows <= 0 || d_ff <= 0) return 0;
  Carver c(nullptr);
  carve_ffn(c, max_rows, d_ff, dtype);
  return c.size();
}

extern "C" int luffy_expert_ffn(const void* x, const int32_t* row_index,
                                const int32_t* rep_offsets, int E, int d, int d_ff,
                                int dtype, const void* w1, const void* w2, int act,
                                int max_rows, void* y_rep,
                                void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !rep_offsets || !w1 || !w2 || !y_rep)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn: null pointer argument");
  if (E <= 0 || d <= 0 || d_ff <= 0 || max_rows <= 0)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn: E=%d d=%d d_ff=%d max_rows=%d", E, d, d_ff, max_rows);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn: unknown dtype %d", dtype);
  if (act != LUFFY_ACT_GELU && act != LUFFY_ACT_SILU)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn: unknown activation %d", act);
  if (E > kMaxExperts) return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn: E=%d > %d", E, kMaxExperts);
  if (d % 64 != 0 || d_ff % 64 != 0)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn: d=%d d_ff=%d must be multiples of 64", d, d_ff);
  if (d > 32768 || d_ff > 32768)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn: d=%d d_ff=%d must be at most 32768", d, d_ff);
  if (static_cast<long long>(max_rows) * d_ff * elem_bytes(dtype) > 0xFFFF0000ll ||
      static_cast<long long>(d) * d_ff * elem_bytes(dtype) > 0xFFFF0000ll)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn: hidden activations or one expert's weights exceed 4 GiB - 64 KiB");
  const size_t need = luffy_expert_ffn_workspace_size(max_rows, E, d_ff, dtype);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_expert_ffn: workspace needs %zu bytes, 256-aligned", need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  const FfnWs ws = carve_ffn(c, max_rows, d_ff, dtype);
  if (act == LUFFY_ACT_GELU)
    launch_ffn<LUFFY_ACT_GELU>(x, row_index, rep_offsets, E, d, d_ff, dtype, w1, w2, max_rows, y_rep, ws, s);
  else
    launch_ffn<LUFFY_ACT_SILU>(x, row_index, rep_offsets, E, d, d_ff, dtype, w1, w2, max_rows, y_rep, ws, s);
  return check_launch("luffy_expert_ffn");
}

extern "C" size_t luffy_expert_ffn_backward_workspace_size(int max_rows, int E, int d, int d_ff, int dtype) {
  if (max_rows <= 0 || E <= 0 || d <= 0 || d_ff <= 0 || dtype != LUFFY_BF16) return 0;
  Carver c(nullptr);
  carve_ffn_bwd(c, max_rows, E, d, d_ff);
  return c.size();
}

extern "C" int luffy_expert_ffn_backward(const void* x, const int32_t* row_index, const int32_t* rep_offsets, int E,
                                         int d, int d_ff, int dtype, const void* w1, const void* w2, int act,
                                         int max_rows, const void* dy_rep, void* dx_rep, void* dw1, void* dw2,
                                         int dw_dtype, void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !rep_offsets || !w1 || !w2 || !dy_rep || !dx_rep || !dw1 || !dw2)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn_backward: null pointer argument");
  if (E <= 0 || d <= 0 || d_ff <= 0 || max_rows <= 0)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn_backward: E=%d d=%d d_ff=%d max_rows=%d", E, d, d_ff, max_rows);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn_backward: unknown dtype %d", dtype);
  if (act != LUFFY_ACT_GELU && act != LUFFY_ACT_SILU)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn_backward: unknown activation %d", act);
  if (dw_dtype != LUFFY_F32 && dw_dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_expert_ffn_backward: unknown weight-gradient dtype %d", dw_dtype);
  if (dtype != LUFFY_BF16) return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn_backward: bf16 only");
  if (E > kMaxExperts) return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn_backward: E=%d > %d", E, kMaxExperts);
  if (d % 64 != 0 || d_ff % 64 != 0)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn_backward: d=%d d_ff=%d must be multiples of 64", d, d_ff);
  if (d > 32768 || d_ff > 32768)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn_backward: d=%d d_ff=%d must be at most 32768", d, d_ff);
  // K-major reads of the activations run up to 63 rows past an expert's last
  const long long krows = static_cast<long long>(max_rows) + 64;
  if (static_cast<long long>(max_rows) * d_ff * 2 > 0xFFFF0000ll ||
      static_cast<long long>(d) * d_ff * 2 > 0xFFFF0000ll ||
      krows * (d > d_ff ? d : d_ff) * 2 > 0xFFFF0000ll)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_expert_ffn_backward: an operand exceeds 4 GiB - 64 KiB");
  const size_t need = luffy_expert_ffn_backward_workspace_size(max_rows, E, d, d_ff, dtype);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_expert_ffn_backward: workspace needs %zu bytes, 256-aligned", need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  const FfnBwdWs ws = carve_ffn_bwd(c, max_rows, E, d, d_ff);
  const auto* xb = static_cast<const uint16_t*>(x);
  const auto* w1b = static_cast<const uint16_t*>(w1);
  const auto* w2b = static_cast<const uint16_t*>(w2);
  const auto* dyb = static_cast<const uint16_t*>(dy_rep);
  auto* dxb = static_cast<uint16_t*>(dx_rep);
  if (act == LUFFY_ACT_GELU)
    launch_ffn_bwd<LUFFY_ACT_GELU>(xb, row_index, rep_offsets, E, d, d_ff, w1b, w2b, max_rows, dyb, dxb, dw1, dw2,
                                   dw_dtype == LUFFY_BF16, ws, s);
  else
    launch_ffn_bwd<LUFFY_ACT_SILU>(xb, row_index, rep_offsets, E, d, d_ff, w1b, w2b, max_rows, dyb, dxb, dw1, dw2,
                                   dw_dtype == LUFFY_BF16, ws, s);
  return check_launch("luffy_expert_ffn_backward");
}

