// luffy_route: gate logits, top-k, gates and the stable dispatch order.
//
// Kernels (all on the caller's stream, no host synchronisation):
//   gate_kernel      64 tokens per block.  bf16: the four waves split the
//                    contraction over d and each accumulates a 64 x E logit
//                    tile on MFMA (16x16x32); fp32: plain FMA.  Top-k, gates
//                    and the float64 re-decision of close calls follow in
//                    the epilogue.
//   slot_hist_kernel 1024 slots per block in slot-id order: stable rank of
//                    every slot among the block's slots of its expert
//                    (wave ballots) and the per-block expert counts.
//   slot_scan_kernel one block: exclusive scan of the block counts per
//                    expert, capacity clamp, bucket offsets.
//   slot_scatter_kernel  bucket position of every slot, capacity drop,
//                    perm_token.
#include <cmath>

#include "luffy_common.h"

namespace luffy {
namespace {

constexpr int kGateTok = 64;     // tokens per gate block
constexpr int kSlotChunk = 1024; // slots per histogram block

template <bool BF16>
__device__ __forceinline__ double elem_f64(const void* base, size_t i) {
  if constexpr (BF16) {
    return static_cast<double>(bf16_to_f32(static_cast<const uint16_t*>(base)[i]));
  } else {
    return static_cast<double>(static_cast<const float*>(base)[i]);
  }
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  // xor butterfly: every lane ends with the same, bit-identical sum
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <bool BF16>
__global__ __launch_bounds__(256) void gate_kernel(
    const void* __restrict__ xv, const void* __restrict__ wv,
    const float* __restrict__ bias, int T, int d, int E, int k,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_gate) {
  __shared__ float part[4][kGateTok][kMaxExperts + 1];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int t0 = blockIdx.x * kGateTok;

  if constexpr (BF16) {
    const uint16_t* X = static_cast<const uint16_t*>(xv);
    const uint16_t* W = static_cast<const uint16_t*>(wv);
    const int nE16 = (E + 15) >> 4;
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint16_t* arow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int t = t0 + 16 * i + (lane & 15);
      t = t < T ? t : T - 1;
      arow[i] = X + static_cast<size_t>(t) * d + 8 * (lane >> 4);
    }
    const uint16_t* brow[4];
    bool bval[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = 16 * j + (lane & 15);
      bval[j] = e < E;
      brow[j] = W + static_cast<size_t>(bval[j] ? e : 0) * d + 8 * (lane >> 4);
    }
    for (int k0 = w * 64; k0 < d; k0 += 256) {
      Pack16 a[4][2], b[4][2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          a[i][h].u4 = *reinterpret_cast<const uint4*>(arow[i] + k0 + 32 * h);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (j < nE16 && bval[j])
            b[j][h].u4 = *reinterpret_cast<const uint4*>(brow[j] + k0 + 32 * h);
          else
            b[j][h].u4 = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (j < nE16) acc[i][j] = mfma16x16x32(a[i][h].v, b[j][h].v, acc[i][j]);
    }
    // lane holds logits of tokens 16i + 4(lane/16) + r, expert 16j + lane%16
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (j < nE16)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            part[w][16 * i + 4 * (lane >> 4) + r][16 * j + (lane & 15)] = acc[i][j][r];
  } else {
    // float32 inputs: one token per lane, experts strided over the waves
    const float* X = static_cast<const float*>(xv);
    const float* W = static_cast<const float*>(wv);
    int t = t0 + lane;
    t = t < T ? t : T - 1;
    for (int e = w; e < E; e += 4) {
      float s = 0.f;
      for (int i = 0; i < d; ++i) s = fmaf(X[static_cast<size_t>(t) * d + i], W[static_cast<size_t>(e) * d + i], s);
      part[0][lane][e] = s;
      part[1][lane][e] = 0.f;
      part[2][lane][e] = 0.f;
      part[3][lane][e] = 0.f;
    }
  }
  __syncthreads();
  if (w != 0) return;

  // ---- epilogue: lane = token
  const int t = t0 + lane;
  const bool valid = t < T;
  const float NEG = -INFINITY;
  float v0 = NEG, v1 = NEG, v2 = NEG;
  int i0 = 0, i1 = 0;
  for (int e = 0; e < E; ++e) {
    float v = part[0][lane][e] + part[1][lane][e] + part[2][lane][e] + part[3][lane][e];
    if (bias) v += bias[e];
    part[0][lane][e] = v;
    if (v > v0) { v2 = v1; v1 = v0; i1 = i0; v0 = v; i0 = e; }
    else if (v > v1) { v2 = v1; v1 = v; i1 = e; }
    else if (v > v2) { v2 = v; }
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
    for (int e = 0; e < E; ++e)
      if (part[0][lane][e] >= vk1 - delta) cand |= 1ull << e;
  uint64_t ambmask = __ballot(amb);
  while (ambmask) {
    const int tl = __ffsll(static_cast<long long>(ambmask)) - 1;
    ambmask &= ambmask - 1;
    const uint64_t cm = static_cast<uint64_t>(__shfl(static_cast<long long>(cand), tl, 64));
    const size_t xt = static_cast<size_t>(t0 + tl) * d;
    double b0 = -INFINITY, b1 = -INFINITY;
    int j0 = 0, j1 = 0;
    for (int e = 0; e < E; ++e) {
      if (!((cm >> e) & 1ull)) continue;
      double s = 0.0;
      for (int i = lane; i < d; i += 64)
        s += elem_f64<BF16>(xv, xt + i) * elem_f64<BF16>(wv, static_cast<size_t>(e) * d + i);
      s = wave_sum_f64(s);
      if (bias) s += static_cast<double>(bias[e]);
      if (s > b0) { b1 = b0; j1 = j0; b0 = s; j0 = e; }
      else if (s > b1) { b1 = s; j1 = e; }
    }
    if (lane == tl) { i0 = j0; i1 = j1; }
  }
  if (!valid) return;
  float den = 0.f;
  for (int e = 0; e < E; ++e) den += expf(part[0][lane][e] - v0);
  if (k == 1) {
    topk_idx[t] = i0;
    topk_gate[t] = expf(part[0][lane][i0] - v0) / den;
  } else {
    const float ga = expf(part[0][lane][i0] - v0);
    const float gb = expf(part[0][lane][i1] - v0);
    topk_idx[2 * t] = i0;
    topk_idx[2 * t + 1] = i1;
    topk_gate[2 * t] = ga / (ga + gb);
    topk_gate[2 * t + 1] = gb / (ga + gb);
  }
}

// Rank of every slot among the slots of the same expert in its 1024-slot
// block (slot id order), and the block's per-expert counts.
__global__ __launch_bounds__(1024) void slot_hist_kernel(
    const int32_t* __restrict__ topk_idx, int T, int k, int E,
    int32_t* __restrict__ slot_rank, int32_t* __restrict__ hist) {
  __shared__ int cnt[16][kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int i = tid; i < 16 * kMaxExperts; i += 1024) (&cnt[0][0])[i] = 0;
  __syncthreads();
  const long long s = static_cast<long long>(blockIdx.x) * kSlotChunk + tid;
  const long long S = static_cast<long long>(T) * k;
  int e = -1, t = 0, j = 0;
  if (s < S) {
    j = static_cast<int>(s / T);
    t = static_cast<int>(s - static_cast<long long>(j) * T);
    e = topk_idx[static_cast<size_t>(t) * k + j];
  }
  const int key = e < 0 ? 127 : e;
  uint64_t same = ~0ull;
#pragma unroll
  for (int b = 0; b < 7; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t bb = __ballot(bit);
    same &= bit ? bb : ~bb;
  }
  const int rank = __popcll(same & lanemask_lt());
  if (e >= 0 && rank == 0) cnt[wv][e] = __popcll(same);
  __syncthreads();
  if (tid < E) {
    int run = 0;
    for (int w2 = 0; w2 < 16; ++w2) {
      const int c = cnt[w2][tid];
      cnt[w2][tid] = run;
      run += c;
    }
    hist[static_cast<size_t>(blockIdx.x) * E + tid] = run;
  }
  __syncthreads();
  if (e >= 0) slot_rank[static_cast<size_t>(t) * k + j] = cnt[wv][e] + rank;
}

// One block: per-expert exclusive scan of the block counts (in place, they
// become block bases), capacity clamp and bucket offsets.
__global__ __launch_bounds__(1024) void slot_scan_kernel(
    int32_t* __restrict__ hist, int nch, int E, int C, int32_t* __restrict__ offsets) {
  constexpr int kLds = 8192;
  __shared__ int buf[kLds];
  __shared__ int run[kMaxExperts];
  const int tid = threadIdx.x;
  if (tid < E) run[tid] = 0;
  const int rows_per_piece = kLds / E;
  for (int c0 = 0; c0 < nch; c0 += rows_per_piece) {
    const int rows = min(rows_per_piece, nch - c0);
    __syncthreads();
    for (int i = tid; i < rows * E; i += 1024) buf[i] = hist[static_cast<size_t>(c0) * E + i];
    __syncthreads();
    if (tid < E) {
      int r = run[tid];
      for (int c = 0; c < rows; ++c) {
        const int v = buf[c * E + tid];
        buf[c * E + tid] = r;
        r += v;
      }
      run[tid] = r;
    }
    __syncthreads();
    for (int i = tid; i < rows * E; i += 1024) hist[static_cast<size_t>(c0) * E + i] = buf[i];
  }
  __syncthreads();
  if (tid == 0) {
    int o = 0;
    for (int e = 0; e < E; ++e) {
      offsets[e] = o;
      const int n = run[e];
      o += (C > 0 && n > C) ? C : n;
    }
    offsets[E] = o;
  }
}

__global__ __launch_bounds__(256) void slot_scatter_kernel(
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ base,
    const int32_t* __restrict__ offsets, int T, int k, int E, int C,
    int32_t* __restrict__ slot_pos, int32_t* __restrict__ perm_token) {
  const long long s = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
  if (s >= static_cast<long long>(T) * k) return;
  const int j = static_cast<int>(s / T);
  const int t = static_cast<int>(s - static_cast<long long>(j) * T);
  const size_t o = static_cast<size_t>(t) * k + j;
  const int e = topk_idx[o];
  const int pos = base[static_cast<size_t>(s / kSlotChunk) * E + e] + slot_pos[o];
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
};

RouteWs carve_route(Carver& c, int T, int E, int k) {
  RouteWs w;
  const long long S = static_cast<long long>(T) * k;
  const long long nch = (S + kSlotChunk - 1) / kSlotChunk;
  w.hist = c.take<int32_t>(static_cast<size_t>(nch) * E);
  return w;
}

}  // namespace

int capacity_slots(int T, int k, int E, float cf) {
  if (!(cf > 0.f)) return 0;
  return static_cast<int>(std::ceil(static_cast<double>(cf) * k * T / E - 1e-9));
}

}  // namespace luffy

using namespace luffy;

extern "C" size_t luffy_route_workspace_size(int T, int E, int k) {
  if (T <= 0 || E <= 0 || k <= 0) return 0;
  Carver c(nullptr);
  carve_route(c, T, E, k);
  return c.size();
}

extern "C" int luffy_route(const void* x, int T, int d, int dtype,
                           const void* w_gate, const float* b_gate, int E, int k,
                           float capacity_factor,
                           int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                           int32_t* perm_token, int32_t* offsets,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !w_gate || !topk_idx || !topk_gate || !slot_pos || !perm_token || !offsets)
    return fail(LUFFY_E_INVALID, "luffy_route: null pointer argument");
  if (T <= 0 || d <= 0 || E <= 0)
    return fail(LUFFY_E_INVALID, "luffy_route: T=%d d=%d E=%d must be positive", T, d, E);
  if (k != 1 && k != 2)
    return fail(LUFFY_E_INVALID, "luffy_route: k=%d must be 1 or 2", k);
  if (k > E) return fail(LUFFY_E_INVALID, "luffy_route: k=%d > E=%d", k, E);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_route: unknown dtype %d", dtype);
  if (E > kMaxExperts)
    return fail(LUFFY_E_UNSUPPORTED, "luffy_route: E=%d > %d", E, kMaxExperts);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_route: d=%d not a multiple of 64", d);
  if (static_cast<long long>(T) * k >= (1ll << 31))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_route: T*k too large");
  const size_t need = luffy_route_workspace_size(T, E, k);
  if (workspace_bytes < need || (need && !workspace) ||
      (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_route: workspace needs %zu bytes, 256-aligned", need);

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  RouteWs ws = carve_route(c, T, E, k);
  const int C = capacity_slots(T, k, E, capacity_factor);
  const long long S = static_cast<long long>(T) * k;
  const int nch = static_cast<int>((S + kSlotChunk - 1) / kSlotChunk);

  const int gblocks = (T + kGateTok - 1) / kGateTok;
  {
    ProfileScope prof_("gate", s);
    if (dtype == LUFFY_BF16)
      gate_kernel<true><<<gblocks, 256, 0, s>>>(x, w_gate, b_gate, T, d, E, k, topk_idx, topk_gate);
    else
      gate_kernel<false><<<gblocks, 256, 0, s>>>(x, w_gate, b_gate, T, d, E, k, topk_idx, topk_gate);
  }
  {
    ProfileScope prof_("slot_hist", s);
    slot_hist_kernel<<<nch, 1024, 0, s>>>(topk_idx, T, k, E, slot_pos, ws.hist);
  }
  {
    ProfileScope prof_("slot_scan", s);
    slot_scan_kernel<<<1, 1024, 0, s>>>(ws.hist, nch, E, C, offsets);
  }
  {
    ProfileScope prof_("slot_scatter", s);
    slot_scatter_kernel<<<static_cast<int>((S + 255) / 256), 256, 0, s>>>(
        topk_idx, ws.hist, offsets, T, k, E, C, slot_pos, perm_token);
  }
  return check_launch("luffy_route");
}
