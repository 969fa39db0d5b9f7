// luffy_route: gate logits, top-k, gates and the stable dispatch order.
//
// Kernels (all on the caller's stream, no host synchronisation):
//   gate_kernel      32 or 64 tokens per block; the four waves split the
//                    contraction over d and accumulate tokens x E logit tiles
//                    on MFMA (16x16x32); fp32: plain FMA.  The epilogue
//                    takes top-k, gates and the float64 re-decision of close
//                    calls, then ranks every slot among the block's slots of
//                    the same expert (wave ballots) and writes the block's
//                    per-expert counts.  A chunk is (choice j, block b), and
//                    chunks in (j, b) order are slots in slot-id order.
//   slot_scan_kernel one block per expert: exclusive scan of its chunk
//                    counts; the last block to finish writes the
//                    capacity-clamped bucket offsets.
//   slot_scatter_kernel  bucket position of every slot, capacity drop,
//                    perm_token.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "luffy_common.h"

// Scratch of luffy_route_noalloc (the per-chunk slot counts of one call):
// one copy per GPU for the life of the process.  In host code the name only
// stands for the symbol; kernels get the device address that
// hipGetSymbolAddress returns for the current device.
static constexpr size_t kRouteScratchBytes = 4u << 20;
static __device__ __align__(256) uint8_t route_scratch[kRouteScratchBytes];

namespace luffy {
namespace {

// Tokens per gate block (= slots per chunk of the histogram): 64, or 32
// when 64 would leave most CUs without a block (T below 32768 makes fewer
// than 512 blocks of 64).  Depends on T only, so workspace sizing and the
// launches always agree.
constexpr int kGateTokMax = 64;
inline int gate_tokens(int T) { return T >= 32768 ? 64 : 32; }

__device__ __forceinline__ double wave_sum_f64(double v) {
  // xor butterfly: every lane ends with the same, bit-identical sum
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Float64 re-decision of one token's close call, by the whole wave: the two
// largest exact logits x.w_e + b_e over the candidate experts cm, visited in
// ascending e (the lower expert first among equal values).  Up to four
// candidates at a time: the lane's 16-byte pieces of x are loaded once per
// batch and every candidate's pieces of W are in flight together (the
// latency of a close call, not its arithmetic, is what the launch waits
// for; NC candidates a batch).  wpiece(e, c) returns the 8 weights of
// expert e at columns c..c+7.
// Each candidate's sum takes the same lane partition and butterfly as a
// one-candidate loop, so the values do not depend on the batching.
template <int NC, class WPiece>
__device__ __forceinline__ int2 redecide_bf16_f64(const uint16_t* __restrict__ xr, WPiece wpiece,
                                                  const float* __restrict__ bias, int d, uint64_t cm) {
  const int lane = threadIdx.x & 63;
  double b0 = -INFINITY, b1 = -INFINITY;
  int j0 = 0, j1 = 0;
  while (cm) {
    int ec[NC];
    int nc = 0;
#pragma unroll
    for (int j = 0; j < NC; ++j) ec[j] = 0;
    for (; nc < NC && cm; ++nc) {
      ec[nc] = __ffsll(static_cast<long long>(cm)) - 1;
      cm &= cm - 1;
    }
    double sacc[NC];
#pragma unroll
    for (int j = 0; j < NC; ++j) sacc[j] = 0.0;
    for (int c = lane * 8; c < d; c += 512) {
      Pack16 xa, wa[NC];
      xa.u4 = *reinterpret_cast<const uint4*>(xr + c);
#pragma unroll
      for (int j = 0; j < NC; ++j) wa[j].u4 = j < nc ? wpiece(ec[j], c) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < NC; ++j)
#pragma unroll
        for (int u = 0; u < 8; ++u)
          sacc[j] += static_cast<double>(bf16_to_f32(xa.h[u])) * static_cast<double>(bf16_to_f32(wa[j].h[u]));
    }
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      if (j >= nc) break;
      const double v = wave_sum_f64(sacc[j]) + static_cast<double>(bias ? bias[ec[j]] : 0.f);
      if (v > b0) { b1 = b0; j1 = j0; b0 = v; j0 = ec[j]; }
      else if (v > b1) { b1 = v; j1 = ec[j]; }
    }
  }
  return make_int2(j0, j1);
}

// Epilogue of a gate chunk of TOK tokens starting at t0, once the logit of
// token tl and expert e (bias included) is in LDS at lg[e * (TOK + 4) + tl]: top-k, gates, the float64
// re-decision of close calls; then wave 0 ranks every slot among the chunk's
// slots of the same expert and writes the chunk's per-expert counts.  Called
// by all four waves of the block; ends with the ranking done (no barrier).
template <bool BF16, int TOK>
__device__ __forceinline__ void gate_select(const float* lg, const float* bias, int* cnt,
                                            int (*choice)[2], const void* __restrict__ xv,
                                            const void* __restrict__ wv, int T, int d, int E, int k, int t0,
                                            int ch, int nchunks, int32_t* __restrict__ topk_idx,
                                            float* __restrict__ topk_gate, int32_t* __restrict__ slot_rank,
                                            int32_t* __restrict__ hist) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  {
    // ---- top-k: wave w takes tokens 16w .. 16w+15, four lanes per token
    // (lane = 4*token + sub); lane sub scans experts sub, sub+4, ... and the
    // four sorted top-3 lists are merged with two shuffle steps.  Order:
    // larger logit first, lower expert index first among equal logits.
    const int sub = lane & 3;
    const int tl_ = min(16 * w + (lane >> 2), TOK - 1);
    const int t = t0 + tl_;
    const bool valid = 16 * w < TOK && t < T;
    const float NEG = -INFINITY;
    float v0 = NEG, v1 = NEG, v2 = NEG;
    int i0 = kMaxExperts, i1 = kMaxExperts, i2 = kMaxExperts;
    if (valid) {
      for (int e = sub; e < E; e += 4) {
        const float v = lg[e * (TOK + 4) + tl_];
        if (v > v0) { v2 = v1; i2 = i1; v1 = v0; i1 = i0; v0 = v; i0 = e; }
        else if (v > v1) { v2 = v1; i2 = i1; v1 = v; i1 = e; }
        else if (v > v2) { v2 = v; i2 = e; }
      }
    }
    auto before = [](float va, int ia, float vb, int ib) { return va > vb || (va == vb && ia < ib); };
#pragma unroll
    for (int o = 1; o <= 2; o <<= 1) {
      const float u0 = __shfl_xor(v0, o, 64), u1 = __shfl_xor(v1, o, 64), u2 = __shfl_xor(v2, o, 64);
      const int j0 = __shfl_xor(i0, o, 64), j1 = __shfl_xor(i1, o, 64), j2 = __shfl_xor(i2, o, 64);
      // merge (v0,v1,v2) and (u0,u1,u2), both sorted, keeping the first three
      float a[3] = {v0, v1, v2}, b[3] = {u0, u1, u2};
      int ai[3] = {i0, i1, i2}, bi[3] = {j0, j1, j2};
      float r[3];
      int ri[3];
      int pa = 0, pb = 0;
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        const float av = pa == 0 ? a[0] : (pa == 1 ? a[1] : a[2]);
        const int aix = pa == 0 ? ai[0] : (pa == 1 ? ai[1] : ai[2]);
        const float bv = pb == 0 ? b[0] : (pb == 1 ? b[1] : b[2]);
        const int bix = pb == 0 ? bi[0] : (pb == 1 ? bi[1] : bi[2]);
        const bool ta = before(av, aix, bv, bix);
        r[q] = ta ? av : bv;
        ri[q] = ta ? aix : bix;
        pa += ta ? 1 : 0;
        pb += ta ? 0 : 1;
      }
      v0 = r[0]; v1 = r[1]; v2 = r[2];
      i0 = ri[0]; i1 = ri[1]; i2 = ri[2];
    }
    // A choice is re-decided in float64 when a deciding gap is within the
    // float32 error budget (about 1e-4 relative; the float32 sums here are
    // accurate to ~1e-6).
    const float delta = ldexpf(1.0f + fabsf(v0), -12);
    const float vk1 = (k == 1) ? v0 : v1;     // k-th largest
    const float vk = (k == 1) ? v1 : v2;      // (k+1)-th largest, -inf if none
    const bool amb = valid && ((k == 2 && v0 - v1 <= delta) || (vk1 - vk <= delta));
    uint64_t cand = 0;
    if (amb)
      for (int e = sub; e < E; e += 4)
        if (lg[e * (TOK + 4) + tl_] >= vk1 - delta) cand |= 1ull << e;
    cand |= static_cast<uint64_t>(__shfl_xor(static_cast<long long>(cand), 1, 64));
    cand |= static_cast<uint64_t>(__shfl_xor(static_cast<long long>(cand), 2, 64));
    uint64_t ambmask = __ballot(amb && sub == 0);
    while (ambmask) {
      const int tl = __ffsll(static_cast<long long>(ambmask)) - 1;   // lane 4 * token
      ambmask &= ambmask - 1;
      const uint64_t cm = static_cast<uint64_t>(__shfl(static_cast<long long>(cand), tl, 64));
      const size_t xt = static_cast<size_t>(t0 + min(16 * w + (tl >> 2), TOK - 1)) * d;
      int j0 = 0, j1 = 0;
      if constexpr (BF16) {
        const uint16_t* W = static_cast<const uint16_t*>(wv);
        const int2 jj = redecide_bf16_f64<4>(
            static_cast<const uint16_t*>(xv) + xt,
            [&](int e, int c) { return *reinterpret_cast<const uint4*>(W + static_cast<size_t>(e) * d + c); },
            bias, d, cm);
        j0 = jj.x;
        j1 = jj.y;
      } else {
        double b0 = -INFINITY, b1 = -INFINITY;
        for (int e = 0; e < E; ++e) {
          if (!((cm >> e) & 1ull)) continue;
          double s = 0.0;
          const float* xr = static_cast<const float*>(xv) + xt;
          const float* wr = static_cast<const float*>(wv) + static_cast<size_t>(e) * d;
          for (int c = lane * 4; c < d; c += 256) {
            const float4 xa = *reinterpret_cast<const float4*>(xr + c);
            const float4 wa = *reinterpret_cast<const float4*>(wr + c);
            s += static_cast<double>(xa.x) * wa.x + static_cast<double>(xa.y) * wa.y +
                 static_cast<double>(xa.z) * wa.z + static_cast<double>(xa.w) * wa.w;
          }
          s = wave_sum_f64(s);
          s += static_cast<double>(bias[e]);
          if (s > b0) { b1 = b0; j1 = j0; b0 = s; j0 = e; }
          else if (s > b1) { b1 = s; j1 = e; }
        }
      }
      if ((lane >> 2) == (tl >> 2)) { i0 = j0; i1 = j1; }
    }
    if (valid) {
      // softmax denominator: e^(l - max) by the hardware exp2 (about 1 ulp),
      // each lane over its quarter of the experts, then summed over the four
      constexpr float kLog2e = 1.44269504088896341f;
      float den = 0.f;
      for (int e = sub; e < E; e += 4) den += __builtin_amdgcn_exp2f((lg[e * (TOK + 4) + tl_] - v0) * kLog2e);
      den += __shfl_xor(den, 1, 64);
      den += __shfl_xor(den, 2, 64);
      if (sub == 0) {
        if (k == 1) {
          topk_idx[t] = i0;
          topk_gate[t] = __builtin_amdgcn_exp2f((lg[i0 * (TOK + 4) + tl_] - v0) * kLog2e) / den;
        } else {
          const float ga = __builtin_amdgcn_exp2f((lg[i0 * (TOK + 4) + tl_] - v0) * kLog2e);
          const float gb = __builtin_amdgcn_exp2f((lg[i1 * (TOK + 4) + tl_] - v0) * kLog2e);
          topk_idx[2 * t] = i0;
          topk_idx[2 * t + 1] = i1;
          topk_gate[2 * t] = ga / (ga + gb);
          topk_gate[2 * t + 1] = gb / (ga + gb);
        }
        choice[tl_][0] = i0;
        choice[tl_][1] = i1;
      }
    }
  }
  __syncthreads();
  if (w == 0) {
    const int t = t0 + lane;
    const bool valid = lane < TOK && t < T;
    const int i0 = valid ? choice[lane][0] : 0, i1 = valid ? choice[lane][1] : 0;
    // stable rank of each slot among this chunk's slots of the same expert:
    // lanes holding the same expert are found with 7 ballots on its bits
    int* cw = cnt;
    for (int j = 0; j < k; ++j) {
      const int e = valid ? (j == 0 ? i0 : i1) : -1;
      const int key = e < 0 ? 127 : e;
      uint64_t same = ~0ull;
#pragma unroll
      for (int b = 0; b < 7; ++b) {
        const bool bit = (key >> b) & 1;
        const uint64_t bb = __ballot(bit);
        same &= bit ? bb : ~bb;
      }
      const int rank = __popcll(same & lanemask_lt());
      if (lane < E) cw[lane] = 0;
      __builtin_amdgcn_wave_barrier();
      if (e >= 0 && rank == 0) cw[e] = __popcll(same);
      __builtin_amdgcn_wave_barrier();
      if (lane < E) hist[static_cast<size_t>(lane) * k * nchunks + static_cast<size_t>(j) * nchunks + ch] = cw[lane];
      if (e >= 0) slot_rank[static_cast<size_t>(t) * k + j] = rank;
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// One block of four waves per chunk of 64 tokens.  bf16: wave w takes the
// w-th quarter of the contraction over d and accumulates the 64 x E logits
// of the chunk on MFMA (16x16x32: four 16-token blocks per 16-expert
// block), two K steps' token and weight loads in flight at a time; the four
// partial tiles are added in LDS in a fixed order.  fp32: plain FMA.  Wave 0 then
// runs the epilogue for the chunk (lane = token): top-k, gates, the float64
// re-decision of close calls, and the rank of every slot among the chunk's
// slots of the same expert (wave ballots) with the chunk's per-expert
// counts.  A chunk is (choice j, chunk c), and chunks in (j, c) order are
// slots in slot-id order.  With inv_norm set, the sums of squares of the
// token columns each lane loads are reduced the same way and 1/|x_t| is
// stored for the similarity pass (0 for a zero row).
template <bool BF16, int TOK>
__global__ __launch_bounds__(256) void gate_kernel(
    const void* __restrict__ xv, const void* __restrict__ wv,
    const float* __restrict__ bias_g, int T, int d, int E, int k,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_gate,
    int32_t* __restrict__ slot_rank, int32_t* __restrict__ hist, int* __restrict__ scan_done,
    float* __restrict__ inv_norm) {
  constexpr int kGateA = TOK / 16;   // 16-token MFMA row blocks
  // partial logits of the four waves, expert-major: part[w][e][tl] (the four
  // consecutive tokens an MFMA lane holds are one 16-byte store)
  constexpr int LD = TOK + 4;
  __shared__ __attribute__((aligned(16))) float part[4][kMaxExperts][LD];
  __shared__ float sumsq[4][TOK];
  __shared__ float bias[kMaxExperts];
  __shared__ int cnt[kMaxExperts];
  __shared__ int choice[TOK][2];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int nchunks = gridDim.x;
  const int ch = blockIdx.x;
  const int t0 = ch * TOK;
  if (threadIdx.x < E) bias[threadIdx.x] = bias_g ? bias_g[threadIdx.x] : 0.f;
  if (blockIdx.x == 0 && threadIdx.x == 0) *scan_done = 0;   // armed for slot_scan_kernel

  if constexpr (BF16) {
    const uint16_t* X = static_cast<const uint16_t*>(xv);
    const uint16_t* W = static_cast<const uint16_t*>(wv);
    const int nE16 = (E + 15) >> 4;
    f32x4 acc[kGateA][4];
#pragma unroll
    for (int i = 0; i < kGateA; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint16_t* arow[kGateA];
#pragma unroll
    for (int i = 0; i < kGateA; ++i)
      arow[i] = X + static_cast<size_t>(min(t0 + 16 * i + (lane & 15), T - 1)) * d + 8 * (lane >> 4);
    const uint16_t* brow[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      brow[j] = W + static_cast<size_t>(min(16 * j + (lane & 15), E - 1)) * d + 8 * (lane >> 4);
    const int nsteps = d / 32;
    const int q = (nsteps + 3) / 4;
    const int s_lo = w * q, s_hi = min(nsteps, s_lo + q);
    constexpr int B = 2;   // K steps per batch; the next batch is loaded while one is multiplied
    // sums of squares of the token rows on MFMA: the Gram of a 16-token
    // block with itself, whose diagonal is the rows' squared norms
    f32x4 accsq[kGateA];
#pragma unroll
    for (int i = 0; i < kGateA; ++i) accsq[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    Pack16 a[2][B][kGateA], b[2][B][4];
    auto load = [&](int s0, Pack16 (&aa)[B][kGateA], Pack16 (&bb)[B][4]) {
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int st = s0 + u;
        const bool in = st < s_hi;
#pragma unroll
        for (int i = 0; i < kGateA; ++i)
          aa[u][i].u4 = in ? *reinterpret_cast<const uint4*>(arow[i] + 32 * st) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          bb[u][j].u4 = (in && j < nE16) ? *reinterpret_cast<const uint4*>(brow[j] + 32 * st)
                                         : make_uint4(0, 0, 0, 0);
      }
    };
    auto compute = [&](const Pack16 (&aa)[B][kGateA], const Pack16 (&bb)[B][4]) {
#pragma unroll
      for (int u = 0; u < B; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (j < nE16)
#pragma unroll
            for (int i = 0; i < kGateA; ++i) acc[i][j] = mfma16x16x32(aa[u][i].v, bb[u][j].v, acc[i][j]);
      if (inv_norm) {
#pragma unroll
        for (int u = 0; u < B; ++u)
#pragma unroll
          for (int i = 0; i < kGateA; ++i) accsq[i] = mfma16x16x32(aa[u][i].v, aa[u][i].v, accsq[i]);
      }
    };
    if (s_lo < s_hi) load(s_lo, a[0], b[0]);
    // unrolled by two so that both register sets are indexed statically
    for (int s0 = s_lo; s0 < s_hi; s0 += 2 * B) {
      if (s0 + B < s_hi) load(s0 + B, a[1], b[1]);
      compute(a[0], b[0]);
      if (s0 + B >= s_hi) break;
      if (s0 + 2 * B < s_hi) load(s0 + 2 * B, a[0], b[0]);
      compute(a[1], b[1]);
    }
    if (inv_norm) {
      // element (m, m) of the 16 x 16 Gram sits in lane 16 (m / 4) + m,
      // register m % 4
      const int m = lane & 15;
      if ((m >> 2) == (lane >> 4)) {
#pragma unroll
        for (int i = 0; i < kGateA; ++i) {
          const int r = m & 3;
          const float v = r == 0 ? accsq[i][0] : (r == 1 ? accsq[i][1] : (r == 2 ? accsq[i][2] : accsq[i][3]));
          sumsq[w][16 * i + m] = v;
        }
      }
    }
    // lane holds logits of tokens 16i + 4(lane/16) + r, expert 16j + lane%16
#pragma unroll
    for (int i = 0; i < kGateA; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (j < nE16)
          *reinterpret_cast<f32x4*>(&part[w][16 * j + (lane & 15)][16 * i + 4 * (lane >> 4)]) = acc[i][j];
  } else {
    // float32 inputs: lane = token (lanes past TOK have none), experts
    // strided over the four waves
    const float* X = static_cast<const float*>(xv);
    const float* W = static_cast<const float*>(wv);
    const int t = min(t0 + lane, T - 1);
    for (int e = w; e < E && lane < TOK; e += 4) {
      float s = 0.f;
      for (int i = 0; i < d; ++i) s = fmaf(X[static_cast<size_t>(t) * d + i], W[static_cast<size_t>(e) * d + i], s);
      part[0][e][lane] = s;
      part[1][e][lane] = 0.f;
      part[2][e][lane] = 0.f;
      part[3][e][lane] = 0.f;
    }
    if (inv_norm && lane < TOK) {
      float s = 0.f;
      for (int i = w; i < d; i += 4) s = fmaf(X[static_cast<size_t>(t) * d + i], X[static_cast<size_t>(t) * d + i], s);
      sumsq[w][lane] = s;
    }
  }
  __syncthreads();
  if (inv_norm && threadIdx.x < TOK && t0 + static_cast<int>(threadIdx.x) < T) {
    const float ss = ((sumsq[0][threadIdx.x] + sumsq[1][threadIdx.x]) + sumsq[2][threadIdx.x]) + sumsq[3][threadIdx.x];
    inv_norm[t0 + threadIdx.x] = ss > 0.f ? 1.0f / sqrtf(ss) : 0.f;
  }
  // partial tiles summed in wave order into part[0], one (expert, token)
  // pair per thread at a time
  {
    constexpr int kPerStep = 256 / TOK;
    const int tl = static_cast<int>(threadIdx.x) % TOK;
    for (int e = static_cast<int>(threadIdx.x) / TOK; e < E; e += kPerStep)
      part[0][e][tl] = ((part[0][e][tl] + part[1][e][tl]) + part[2][e][tl]) + part[3][e][tl] + bias[e];
  }
  __syncthreads();
  gate_select<BF16, TOK>(&part[0][0][0], bias, cnt, choice, xv, wv, T, d, E, k, t0, ch, nchunks, topk_idx,
                         topk_gate, slot_rank, hist);
}

// ------------------------------------------------------------ streaming gate
// bf16 gate for a weight matrix of at most kGateLdsW bytes (E <= 64): one
// persistent block of 16 waves per CU stages W in LDS once, and every wave
// then takes chunks of 16 tokens over the whole of d.  A wave keeps eight
// K steps of token loads (8 KB) in flight while it multiplies the previous
// eight, so a CU has ~128 KB of its token stream in flight; the logits stay
// in the MFMA accumulators (lane = expert 16j + lane%16 of tokens
// 4(lane/16) .. +3) and top-k runs on them in place, with row-wide DPP
// reductions over the 16 lanes that hold one token's experts, so nothing
// but the per-chunk slot counts passes through LDS.  A chunk of the slot
// histogram is one wave's 16 tokens.
constexpr int kGateLdsW = 128 * 1024;            // bytes of W held in LDS
constexpr int kGateStreamWaves = 16;
constexpr int kGateStreamTok = 16;               // tokens per chunk (one wave)
constexpr int kGateStreamNB = 4;                 // K steps (of 32) per load batch
constexpr int kGateStreamNC = 1;                 // close-call candidates a batch (no spills)

inline bool gate_stream_ok(int dtype, int E, int d) {
  return dtype == LUFFY_BF16 && E <= kMaxExperts && static_cast<long long>(E) * d * 2 <= kGateLdsW && d % 64 == 0;
}

// rotation by N lanes inside each row of 16 lanes (DPP row_ror)
template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x120 + N, 0xF, 0xF, false));
}
// every lane of a row ends with the maximum (or sum) of the row's 16 values
__device__ __forceinline__ uint32_t row_max_u32(uint32_t x) {
  x = max(x, row_ror<8>(x));
  x = max(x, row_ror<4>(x));
  x = max(x, row_ror<2>(x));
  return max(x, row_ror<1>(x));
}
__device__ __forceinline__ float row_max_f32(float x) {
  x = fmaxf(x, __uint_as_float(row_ror<8>(__float_as_uint(x))));
  x = fmaxf(x, __uint_as_float(row_ror<4>(__float_as_uint(x))));
  x = fmaxf(x, __uint_as_float(row_ror<2>(__float_as_uint(x))));
  return fmaxf(x, __uint_as_float(row_ror<1>(__float_as_uint(x))));
}
__device__ __forceinline__ float row_sum_f32(float x) {
  x += __uint_as_float(row_ror<8>(__float_as_uint(x)));
  x += __uint_as_float(row_ror<4>(__float_as_uint(x)));
  x += __uint_as_float(row_ror<2>(__float_as_uint(x)));
  return x + __uint_as_float(row_ror<1>(__float_as_uint(x)));
}

// Order-preserving key of a logit with the expert in its low six bits: a
// larger key is a larger logit, and among logits equal in their top 26 bits
// the lower expert.  Dropping the low six mantissa bits moves a value by
// less than 2^-17 of itself; every decision closer than the float64
// re-decision margin (2^-11 (1 + |max|), far wider) goes to float64 anyway.
__device__ __forceinline__ uint32_t logit_key(float v, int e) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (o & ~63u) | static_cast<uint32_t>(63 - e);
}
__device__ __forceinline__ float key_value(uint32_t key) {
  if (key == 0u) return -INFINITY;                  // no such expert
  const uint32_t o = key & ~63u;
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ int key_expert(uint32_t key) { return 63 - static_cast<int>(key & 63u); }

template <int NEB>
__global__ __launch_bounds__(kGateStreamWaves * 64) void gate_stream_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, const float* __restrict__ bias_g, int T, int d,
    int E, int k, int nchunks, int32_t* __restrict__ topk_idx, float* __restrict__ topk_gate,
    int32_t* __restrict__ slot_rank, int32_t* __restrict__ hist, int* __restrict__ scan_done,
    float* __restrict__ inv_norm) {
  // W (row e, 16-byte chunk c at e * d/8 + (c ^ (e & 7)): the 16 rows one
  // fragment read touches fall on distinct banks), then 64 slot counts a wave
  __shared__ __attribute__((aligned(16))) uint8_t lds[kGateLdsW + kGateStreamWaves * kMaxExperts * 4];
  uint4* wl = reinterpret_cast<uint4*>(lds);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int m = lane & 15, q = lane >> 4;
  const int cpr = d >> 3;                          // 16-byte chunks per W row
  if (blockIdx.x == 0 && tid == 0) *scan_done = 0;   // armed for slot_scan_kernel
  for (int i = tid; i < E * cpr; i += kGateStreamWaves * 64) {
    const int e = i / cpr, c = i - e * cpr;
    wl[e * cpr + (c ^ (e & 7))] = reinterpret_cast<const uint4*>(W)[i];
  }
  // per expert block j: this lane's W row base, its chunk swizzle folded
  // with the lane's K group, and the expert's bias (-inf past E)
  int brow[NEB], bsw[NEB];
  float bias[NEB];
#pragma unroll
  for (int j = 0; j < NEB; ++j) {
    const int e = 16 * j + m;
    const int er = min(e, E - 1);
    brow[j] = er * cpr;
    bsw[j] = q ^ (er & 7);
    bias[j] = e < E ? (bias_g ? bias_g[e] : 0.f) : -INFINITY;
  }
  int* cw = reinterpret_cast<int*>(lds + kGateLdsW) + w * kMaxExperts;
  __syncthreads();

  const int nsteps = d >> 5;
  constexpr int NB = kGateStreamNB;
  for (int ch = blockIdx.x * kGateStreamWaves + w; ch < nchunks; ch += gridDim.x * kGateStreamWaves) {
    const int t0 = ch * kGateStreamTok;
    const uint16_t* arow = X + static_cast<size_t>(min(t0 + m, T - 1)) * d + 8 * q;
    Pack16 a[2][NB];
    auto load = [&](int s0, Pack16 (&aa)[NB]) {
#pragma unroll
      for (int u = 0; u < NB; ++u)
        aa[u].u4 = s0 + u < nsteps ? *reinterpret_cast<const uint4*>(arow + 32 * (s0 + u)) : make_uint4(0, 0, 0, 0);
    };
    f32x4 acc[NEB];
#pragma unroll
    for (int j = 0; j < NEB; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 accsq = f32x4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int s0, const Pack16 (&aa)[NB]) {
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        if (s0 + u >= nsteps) break;
        const int c4 = 4 * (s0 + u);
#pragma unroll
        for (int j = 0; j < NEB; ++j) {
          Pack16 b;
          b.u4 = wl[brow[j] + (c4 ^ bsw[j])];
          acc[j] = mfma16x16x32(aa[u].v, b.v, acc[j]);
        }
        if (inv_norm) accsq = mfma16x16x32(aa[u].v, aa[u].v, accsq);
      }
    };
    load(0, a[0]);
    for (int s0 = 0; s0 < nsteps; s0 += 2 * NB) {
      if (s0 + NB < nsteps) load(s0 + NB, a[1]);
      compute(s0, a[0]);
      if (s0 + NB >= nsteps) break;
      if (s0 + 2 * NB < nsteps) load(s0 + 2 * NB, a[0]);
      compute(s0 + NB, a[1]);
    }

    // ---- epilogue.  Register i of acc[j] holds token 4q + i, expert
    // 16j + m; the 16 lanes of row q hold all experts of tokens 4q .. 4q+3.
    // Token 4q + i is decided on row q's lanes, then kept by lane 16q + i
    // (lanes in token order).
    const int r = m & 3;
    int c0 = 0, c1 = 0;
    float h0 = 0.f, h1 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t key[NEB];
#pragma unroll
      for (int j = 0; j < NEB; ++j) {
        const float v = acc[j][i] + bias[j];
        acc[j][i] = v;
        key[j] = 16 * j + m < E ? logit_key(v, 16 * j + m) : 0u;
      }
      uint32_t m1 = 0, m2 = 0, m3 = 0;
#pragma unroll
      for (int j = 0; j < NEB; ++j) m1 = max(m1, key[j]);
      m1 = row_max_u32(m1);
#pragma unroll
      for (int j = 0; j < NEB; ++j) m2 = max(m2, key[j] < m1 ? key[j] : 0u);
      m2 = row_max_u32(m2);
      if (k == 2) {
#pragma unroll
        for (int j = 0; j < NEB; ++j) m3 = max(m3, key[j] < m2 ? key[j] : 0u);
        m3 = row_max_u32(m3);
      }
      const float v0 = key_value(m1), v1 = key_value(m2), v2 = key_value(m3);
      // v0 is within 2^-17 of the largest logit: the softmax shift and the
      // scale of the margin
      const float vm = v0;
      const float delta = ldexpf(1.0f + fabsf(vm), -11);
      const bool amb = (v0 - v1 <= delta) || (k == 2 && v1 - v2 <= delta);
      const float thr = (k == 1 ? v0 : v1) - delta;
      int e0 = key_expert(m1), e1 = key_expert(m2);
      // close calls re-decided in float64 from the exact bf16 products over
      // the experts within the margin of the k-th logit (rare; a
      // wave-uniform loop over the row leaders, bit 16q = row q)
      uint64_t ambmask = __ballot(amb && m == 0 && t0 + 4 * q + i < T);
      while (ambmask) {
        const int b = __ffsll(static_cast<long long>(ambmask)) - 1;
        ambmask &= ambmask - 1;
        const int qq = b >> 4;
        uint64_t cm = 0;
#pragma unroll
        for (int j = 0; j < NEB; ++j) {
          const uint64_t bl = __ballot(16 * j + m < E && acc[j][i] >= thr);
          cm |= ((bl >> (16 * qq)) & 0xFFFFull) << (16 * j);
        }
        const int2 jj = redecide_bf16_f64<kGateStreamNC>(
            X + static_cast<size_t>(t0 + 4 * qq + i) * d,
            [&](int e, int c) { return wl[e * cpr + ((c >> 3) ^ (e & 7))]; }, bias_g, d, cm);
        const int j0 = jj.x, j1 = jj.y;
        if (q == qq) { e0 = j0; e1 = j1; }
      }
      // gates from the float32 logits of the chosen experts
      constexpr float kLog2e = 1.44269504088896341f;
      float l0 = -INFINITY, l1 = -INFINITY, den = 0.f;
#pragma unroll
      for (int j = 0; j < NEB; ++j) {
        const int e = 16 * j + m;
        l0 = e == e0 ? acc[j][i] : l0;
        l1 = e == e1 ? acc[j][i] : l1;
        if (k == 1) den += __builtin_amdgcn_exp2f((acc[j][i] - vm) * kLog2e);
      }
      l0 = row_max_f32(l0);
      float g0, g1 = 0.f;
      if (k == 1) {
        den = row_sum_f32(den);
        g0 = __builtin_amdgcn_exp2f((l0 - vm) * kLog2e) / den;
      } else {
        l1 = row_max_f32(l1);
        const float ga = __builtin_amdgcn_exp2f((l0 - vm) * kLog2e);
        const float gb = __builtin_amdgcn_exp2f((l1 - vm) * kLog2e);
        g0 = ga / (ga + gb);
        g1 = gb / (ga + gb);
      }
      if (r == i) { c0 = e0; c1 = e1; h0 = g0; h1 = g1; }
    }
    const int tl = 4 * q + m;
    const int t = t0 + tl;
    const bool valid = m < 4 && t < T;
    if (valid) {
      if (k == 1) {
        topk_idx[t] = c0;
        topk_gate[t] = h0;
      } else {
        topk_idx[2 * t] = c0;
        topk_idx[2 * t + 1] = c1;
        topk_gate[2 * t] = h0;
        topk_gate[2 * t + 1] = h1;
      }
    }
    if (inv_norm) {
      // element (mm, mm) of the 16 x 16 Gram: lane 16 (mm / 4) + mm, register mm % 4
      if ((m >> 2) == q && t0 + m < T) {
        const float ss = r == 0 ? accsq[0] : (r == 1 ? accsq[1] : (r == 2 ? accsq[2] : accsq[3]));
        inv_norm[t0 + m] = ss > 0.f ? 1.0f / sqrtf(ss) : 0.f;
      }
    }
    // stable rank of each slot among the chunk's slots of the same expert
    // (7 ballots on the expert bits) and the chunk's per-expert counts
    for (int j = 0; j < k; ++j) {
      const int e = valid ? (j == 0 ? c0 : c1) : -1;
      const int key = e < 0 ? 127 : e;
      uint64_t same = ~0ull;
#pragma unroll
      for (int b = 0; b < 7; ++b) {
        const bool bit = (key >> b) & 1;
        const uint64_t bb = __ballot(bit);
        same &= bit ? bb : ~bb;
      }
      const int rank = __popcll(same & lanemask_lt());
      if (lane < E) cw[lane] = 0;
      __builtin_amdgcn_wave_barrier();
      if (e >= 0 && rank == 0) cw[e] = __popcll(same);
      __builtin_amdgcn_wave_barrier();
      if (lane < E) hist[static_cast<size_t>(lane) * k * nchunks + static_cast<size_t>(j) * nchunks + ch] = cw[lane];
      if (e >= 0) slot_rank[static_cast<size_t>(t) * k + j] = rank;
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// One block per expert: exclusive scan of that expert's chunk counts (in
// place, they become chunk bases) and its total.  The last block to finish
// (a counter, no waiting) turns the totals into capacity-clamped bucket
// offsets and re-arms the counter for the next call.
__global__ __launch_bounds__(1024) void slot_scan_kernel(
    int32_t* __restrict__ hist, int nch, int E, int C, int32_t* __restrict__ offsets,
    int* __restrict__ totals, int* __restrict__ done) {
  __shared__ int wsum[16];
  __shared__ bool last;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int e = blockIdx.x;
  // the expert's counts are contiguous (expert-major layout); each thread
  // takes four consecutive chunks per pass of 4096
  int32_t* h = hist + static_cast<size_t>(e) * nch;
  int carry = 0;
  for (int c0 = 0; c0 < nch; c0 += 4096) {
    const int c = c0 + 4 * tid;
    int v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = c + u < nch ? h[c + u] : 0;
    const int own = (v[0] + v[1]) + (v[2] + v[3]);
    int incl = own;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
      const int u = __shfl_up(incl, sh, 64);
      if (lane >= sh) incl += u;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int wb = 0, tot = 0;
    for (int i = 0; i < 16; ++i) {
      wb += i < wv ? wsum[i] : 0;
      tot += wsum[i];
    }
    int run = carry + wb + incl - own;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (c + u < nch) h[c + u] = run;
      run += v[u];
    }
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) {
    store_flag(&totals[e], carry);
    __threadfence();
    last = atomicAdd(done, 1) == E - 1;
  }
  __syncthreads();
  if (last && wv == 0) {
    // capacity-clamped totals, one expert per lane (E <= 64), prefixed
    __threadfence();
    int n = lane < E ? load_flag(&totals[lane]) : 0;
    if (C > 0 && n > C) n = C;
    int incl = n;
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
      const int u = __shfl_up(incl, sh, 64);
      if (lane >= sh) incl += u;
    }
    if (lane < E) offsets[lane] = incl - n;
    if (lane == E - 1) offsets[E] = incl;
    if (lane == 0) store_flag(done, 0);
  }
}

__global__ __launch_bounds__(256) void slot_scatter_kernel(
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ base,
    const int32_t* __restrict__ offsets, int T, int k, int E, int C, int tok,
    int32_t* __restrict__ slot_pos, int32_t* __restrict__ perm_token) {
  const long long s = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
  if (s >= static_cast<long long>(T) * k) return;
  const int j = static_cast<int>(s / T);
  const int t = static_cast<int>(s - static_cast<long long>(j) * T);
  const size_t o = static_cast<size_t>(t) * k + j;
  const int e = topk_idx[o];
  const int nblk = (T + tok - 1) / tok;
  const int pos = base[static_cast<size_t>(e) * k * nblk + static_cast<size_t>(j) * nblk + t / tok] + slot_pos[o];
  if (C > 0 && pos >= C) {
    slot_pos[o] = -1;
  } else {
    const int p = offsets[e] + pos;
    slot_pos[o] = p;
    perm_token[p] = t;
  }
}

struct RouteWs {
  int32_t* hist;
  int* totals;
  int* done;
};

RouteWs carve_route(Carver& c, int T, int E, int k) {
  RouteWs w;
  // sized for the smallest chunk of either gate kernel
  const long long nch = static_cast<long long>(k) * ((T + kGateStreamTok - 1) / kGateStreamTok);
  w.hist = c.take<int32_t>(static_cast<size_t>(nch) * E);
  w.totals = c.take<int>(E);
  w.done = c.take<int>(1);
  return w;
}

}  // namespace

// ceil(cf*k*T/E - 1e-9) in double precision, evaluated left to right; the
// 1e-9 keeps a product that is an integer up to the rounding of a decimal
// factor (cf = 1.1, k*T/E = 1000) at that integer.
int capacity_slots(int T, int k, int E, double cf) {
  if (!(cf > 0.0)) return 0;
  const double c = std::ceil(cf * k * T / E - 1e-9);
  return c >= 2147483647.0 ? 2147483647 : static_cast<int>(c);
}

}  // namespace luffy

using namespace luffy;

extern "C" size_t luffy_route_workspace_size(int T, int E, int k) {
  if (T <= 0 || E <= 0 || k <= 0) return 0;
  Carver c(nullptr);
  carve_route(c, T, E, k);
  return c.size();
}

namespace {

// Host checks shared by both route entry points.
int route_check(const char* fn, const void* x, int T, int d, int dtype, const void* w_gate, int E, int k,
                const int32_t* topk_idx, const float* topk_gate, const int32_t* slot_pos, const int32_t* perm_token,
                const int32_t* offsets) {
  if (!x || !w_gate || !topk_idx || !topk_gate || !slot_pos || !perm_token || !offsets)
    return fail(LUFFY_E_INVALID, "%s: null pointer argument", fn);
  if (T <= 0 || d <= 0 || E <= 0)
    return fail(LUFFY_E_INVALID, "%s: T=%d d=%d E=%d must be positive", fn, T, d, E);
  if (k != 1 && k != 2)
    return fail(LUFFY_E_INVALID, "%s: k=%d must be 1 or 2", fn, k);
  if (k > E) return fail(LUFFY_E_INVALID, "%s: k=%d > E=%d", fn, k, E);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "%s: unknown dtype %d", fn, dtype);
  if (E > kMaxExperts)
    return fail(LUFFY_E_UNSUPPORTED, "%s: E=%d > %d", fn, E, kMaxExperts);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "%s: d=%d not a multiple of 64", fn, d);
  if (static_cast<long long>(T) * k >= (1ll << 31))
    return fail(LUFFY_E_UNSUPPORTED, "%s: T*k too large", fn);
  return LUFFY_OK;
}

// The three launches of a route call on scratch `ws`.
void route_enqueue(const void* x, int T, int d, int dtype, const void* w_gate, const float* b_gate, int E, int k,
                   double capacity_factor, int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                   int32_t* perm_token, int32_t* offsets, float* inv_norm, const RouteWs& ws, hipStream_t s) {
  const int C = capacity_slots(T, k, E, capacity_factor);
  const long long S = static_cast<long long>(T) * k;
  // the streaming gate when every wave of its persistent grid has a chunk
  const bool stream = gate_stream_ok(dtype, E, d) &&
                      (T + kGateStreamTok - 1) / kGateStreamTok >= kGateStreamWaves * persistent_grid();
  const int tok = stream ? kGateStreamTok : gate_tokens(T);
  const int gblocks = (T + tok - 1) / tok;
  const int nch = k * gblocks;
  if (stream) {
    const int grid = std::max(1, std::min(persistent_grid(), (gblocks + kGateStreamWaves - 1) / kGateStreamWaves));
#define LUFFY_GATE_S(NEB) launch("gate", gate_stream_kernel<NEB>, grid, kGateStreamWaves * 64, 0, s,                  \
                                 static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_gate), b_gate, T, d, \
                                 E, k, gblocks, topk_idx, topk_gate, slot_pos, ws.hist, ws.done, inv_norm)
    if (E <= 16) LUFFY_GATE_S(1);
    else if (E <= 32) LUFFY_GATE_S(2);
    else if (E <= 48) LUFFY_GATE_S(3);
    else LUFFY_GATE_S(4);
#undef LUFFY_GATE_S
  } else {
#define LUFFY_GATE_ARGS x, w_gate, b_gate, T, d, E, k, topk_idx, topk_gate, slot_pos, ws.hist, ws.done, inv_norm
    if (dtype == LUFFY_BF16) {
      if (tok == 32) launch("gate", gate_kernel<true, 32>, gblocks, 256, 0, s, LUFFY_GATE_ARGS);
      else launch("gate", gate_kernel<true, kGateTokMax>, gblocks, 256, 0, s, LUFFY_GATE_ARGS);
    } else {
      if (tok == 32) launch("gate", gate_kernel<false, 32>, gblocks, 256, 0, s, LUFFY_GATE_ARGS);
      else launch("gate", gate_kernel<false, kGateTokMax>, gblocks, 256, 0, s, LUFFY_GATE_ARGS);
    }
#undef LUFFY_GATE_ARGS
  }
  launch("slot_scan", slot_scan_kernel, E, 1024, 0, s, ws.hist, nch, E, C, offsets, ws.totals, ws.done);
  launch("slot_scatter", slot_scatter_kernel, static_cast<int>((S + 255) / 256), 256, 0, s, topk_idx, ws.hist,
         offsets, T, k, E, C, tok, slot_pos, perm_token);
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this GPU's route_scratch, looked up once per device.
int route_scratch_ptr(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(LUFFY_E_HIP, "luffy_route_noalloc: no current device (or device id >= %d)", kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(route_scratch));
    if (e != hipSuccess || !p)
      return fail(LUFFY_E_HIP, "luffy_route_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LUFFY_OK;
}

}  // namespace

extern "C" int luffy_capacity(int T, int k, int E, double capacity_factor) {
  if (T <= 0 || k <= 0 || E <= 0) return 0;
  return capacity_slots(T, k, E, capacity_factor);
}

extern "C" int luffy_route(const void* x, int T, int d, int dtype,
                           const void* w_gate, const float* b_gate, int E, int k,
                           double capacity_factor,
                           int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                           int32_t* perm_token, int32_t* offsets, float* inv_norm,
                           void* workspace, size_t workspace_bytes, void* stream) {
  const int st = route_check("luffy_route", x, T, d, dtype, w_gate, E, k, topk_idx, topk_gate, slot_pos, perm_token,
                             offsets);
  if (st != LUFFY_OK) return st;
  const size_t need = luffy_route_workspace_size(T, E, k);
  if (workspace_bytes < need || (need && !workspace) ||
      (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_route: workspace needs %zu bytes, 256-aligned", need);
  Carver c(workspace);
  const RouteWs ws = carve_route(c, T, E, k);
  route_enqueue(x, T, d, dtype, w_gate, b_gate, E, k, capacity_factor, topk_idx, topk_gate, slot_pos, perm_token,
                offsets, inv_norm, ws, static_cast<hipStream_t>(stream));
  return check_launch("luffy_route");
}

extern "C" size_t luffy_route_noalloc_max_bytes(void) { return kRouteScratchBytes; }

extern "C" int luffy_route_noalloc(const void* x, int T, int d, int dtype,
                                   const void* w_gate, const float* b_gate, int E, int k,
                                   double capacity_factor,
                                   int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                                   int32_t* perm_token, int32_t* offsets, float* inv_norm, void* stream) {
  const int st = route_check("luffy_route_noalloc", x, T, d, dtype, w_gate, E, k, topk_idx, topk_gate, slot_pos,
                             perm_token, offsets);
  if (st != LUFFY_OK) return st;
  const size_t need = luffy_route_workspace_size(T, E, k);
  if (need > kRouteScratchBytes)
    return fail(LUFFY_E_UNSUPPORTED,
                "luffy_route_noalloc: T=%d E=%d k=%d needs %zu bytes of scratch, more than its %zu", T, E, k, need,
                kRouteScratchBytes);
  void* scratch = nullptr;
  const int sp = route_scratch_ptr(&scratch);
  if (sp != LUFFY_OK) return sp;
  Carver c(scratch);
  const RouteWs ws = carve_route(c, T, E, k);
  route_enqueue(x, T, d, dtype, w_gate, b_gate, E, k, capacity_factor, topk_idx, topk_gate, slot_pos, perm_token,
                offsets, inv_norm, ws, static_cast<hipStream_t>(stream));
  return check_launch("luffy_route_noalloc");
}
