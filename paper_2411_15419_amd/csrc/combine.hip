// luffy_combine: y[t] = sum over kept slots j of gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
// One wave per token; 16-byte vector loads and stores (four per lane in
// flight per source row, eight in all); float32 sums.
#include <algorithm>

#include "luffy_common.h"

namespace luffy {
namespace {

// Rows of y_rep are read through a buffer resource: a slot without a
// representative (dropped, or k < 2) and a column chunk past d get the
// out-of-range offset kRange, and robust buffer access returns zeros for
// them.  Every load is therefore unconditional and all of a lane's loads are
// in flight before the first is used (a load behind a branch would wait for
// the one before it).  y_rep must span less than kRange bytes (checked on
// the host against T*k rows).
constexpr uint32_t kRange = 0xFFFF0000u;

// K: slots per token (1 or 2); U: 16-byte chunks per lane per pass (2 when
// two passes' worth of chunks cover a row, else 4), so no load is issued for
// a source or a chunk that cannot exist.
template <bool BF16, int K, int U>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y_rep,
                                                      const int32_t* __restrict__ rep_row,
                                                      const int32_t* __restrict__ slot_pos,
                                                      const float* __restrict__ gate, int T, int d,
                                                      void* __restrict__ y) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int k = K;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  constexpr int ES = BF16 ? 2 : 4;          // bytes per element
  constexpr int EPC = 16 / ES;              // elements per 16-byte chunk
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(y_rep),
                                                                       static_cast<short>(0),
                                                                       static_cast<int>(kRange), 0x00020000);
  uint32_t rbase[2] = {kRange, kRange};
  float g[2] = {0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * k + j];
    if (p >= 0) {
      rbase[j] = static_cast<uint32_t>(rep_row[p]) * static_cast<uint32_t>(d) * ES;
      g[j] = gate[static_cast<size_t>(t) * k + j];
    }
  }
  // U 16-byte chunks per lane per pass
  for (int c0 = lane * EPC; c0 < d; c0 += U * 64 * EPC) {
    u32x4 v[K][U];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * 64 * EPC;
        const uint32_t off = (rbase[j] == kRange || c >= d) ? kRange : rbase[j] + static_cast<uint32_t>(c) * ES;
        v[j][u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 64 * EPC;
      if (c >= d) break;
      if constexpr (BF16) {
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          a[i] = 0.f;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const uint32_t word = v[j][u][i >> 1];
            const float f = __uint_as_float((i & 1) ? (word & 0xFFFF0000u) : (word << 16));
            a[i] = fmaf(g[j], f, a[i]);
          }
        }
        uint16_t* dst = static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d;
        *reinterpret_cast<uint4*>(dst + c) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                                        pack_bf16x2(a[4], a[5]), pack_bf16x2(a[6], a[7]));
      } else {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < K; ++j) {
          a.x = fmaf(g[j], __uint_as_float(v[j][u][0]), a.x);
          a.y = fmaf(g[j], __uint_as_float(v[j][u][1]), a.y);
          a.z = fmaf(g[j], __uint_as_float(v[j][u][2]), a.z);
          a.w = fmaf(g[j], __uint_as_float(v[j][u][3]), a.w);
        }
        float* dst = static_cast<float*>(y) + static_cast<size_t>(t) * d;
        *reinterpret_cast<float4*>(dst + c) = a;
      }
    }
  }
}


// ---------------------------------------------------------------- backward
// Transpose of combine (the condensation held fixed): every kept slot adds
// gate * dy[t] to its representative's row, and takes <dy[t], y_rep[r]> as
// its gate gradient.
//
// Row sums, one work item per (bucket e, range of up to kGatherReps of its
// representatives, 64-column chunk): the item walks the bucket's positions
// 64 at a time (lane = position), and every lane whose position belongs to
// a representative of the range loads its 64 columns of dy (eight 16-byte
// loads, all in flight together) and adds gate * dy into that
// representative's row of an LDS accumulator (LDS float atomics: several
// positions of one group may add at once, so the order of the additions is
// not fixed).  The rows are then rounded into dy_rep.  A bucket's
// representatives are a contiguous range of compact rows
// [rep_offsets[e], rep_offsets[e+1]) and each one's members lie in its own
// bucket, so nothing crosses items and no global atomics are needed.
constexpr int kGatherCols = 64;
constexpr int kGatherReps = 224;   // rows of the LDS accumulator (57 KB with padding)
constexpr int kGatherPitch = kGatherCols + 1;   // padded: lanes on different rows, same column, differ in bank

template <bool BF16, int K>
__global__ __launch_bounds__(256) void cbwd_rows_kernel(const void* __restrict__ dy,
                                                        const int32_t* __restrict__ rep_row,
                                                        const int32_t* __restrict__ perm_token,
                                                        const int32_t* __restrict__ slot_pos,
                                                        const float* __restrict__ gate,
                                                        const int32_t* __restrict__ offsets,
                                                        const int32_t* __restrict__ rep_offsets, int E, int d,
                                                        int max_rows, void* __restrict__ dy_rep) {
  __shared__ float acc[kGatherReps * kGatherPitch];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // work map: lane e < E holds expert e's representative range count
  int m = 0, rlo = 0, rhi = 0, plo = 0, phi = 0;
  if (lane < E) {
    rlo = rep_offsets[lane];
    rhi = rep_offsets[lane + 1];
    plo = offsets[lane];
    phi = offsets[lane + 1];
    m = (rhi - rlo + kGatherReps - 1) / kGatherReps;
  }
  int incl = m;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  const int units = __builtin_amdgcn_readfirstlane(__shfl(incl, 63, 64));
  const int nc = d / kGatherCols;
  const int total = units * nc;
  for (int item = blockIdx.x; item < total; item += gridDim.x) {
    const int u = item / nc, cc = item - u * nc;
    const int e = __popcll(__ballot(lane < E && incl <= u));
    const int excl = __shfl(incl - m, e, 64);
    const int ra = __shfl(rlo, e, 64) + (u - excl) * kGatherReps;
    const int rb = min(ra + kGatherReps, __shfl(rhi, e, 64));
    const int p_lo = __shfl(plo, e, 64), p_hi = __shfl(phi, e, 64);
    for (int i = tid; i < kGatherReps * kGatherPitch; i += 256) acc[i] = 0.f;
    __syncthreads();
    const int c0 = cc * kGatherCols;
    for (int p0 = p_lo + 64 * w; p0 < p_hi; p0 += 256) {
      const int p = p0 + lane;
      const int r = p < p_hi ? rep_row[p] : -1;
      if (r >= ra && r < rb) {
        const int t = perm_token[p];
        const int j = (K == 2 && slot_pos[static_cast<size_t>(t) * K] != p) ? 1 : 0;
        const float g = gate[static_cast<size_t>(t) * K + j];
        float v[kGatherCols];
        if constexpr (BF16) {
          const uint4* src = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(dy) +
                                                            static_cast<size_t>(t) * d + c0);
          uint4 q[kGatherCols / 8];
#pragma unroll
          for (int i = 0; i < kGatherCols / 8; ++i) q[i] = src[i];
#pragma unroll
          for (int i = 0; i < kGatherCols / 8; ++i) {
            const uint32_t wv[4] = {q[i].x, q[i].y, q[i].z, q[i].w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
              v[8 * i + 2 * h] = __uint_as_float(wv[h] << 16);
              v[8 * i + 2 * h + 1] = __uint_as_float(wv[h] & 0xFFFF0000u);
            }
          }
        } else {
          const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(dy) +
                                                              static_cast<size_t>(t) * d + c0);
          float4 q[kGatherCols / 4];
#pragma unroll
          for (int i = 0; i < kGatherCols / 4; ++i) q[i] = src[i];
#pragma unroll
          for (int i = 0; i < kGatherCols / 4; ++i) {
            v[4 * i] = q[i].x;
            v[4 * i + 1] = q[i].y;
            v[4 * i + 2] = q[i].z;
            v[4 * i + 3] = q[i].w;
          }
        }
        float* row = acc + (r - ra) * kGatherPitch;
#pragma unroll
        for (int c = 0; c < kGatherCols; ++c) atomicAdd(row + c, g * v[c]);
      }
    }
    __syncthreads();
    for (int i = tid; i < (rb - ra) * kGatherCols; i += 256) {
      const int rl = i / kGatherCols, c = i - rl * kGatherCols;
      const int r = ra + rl;
      if (r >= max_rows) continue;
      const float a = acc[rl * kGatherPitch + c];
      const size_t o = static_cast<size_t>(r) * d + c0 + c;
      if constexpr (BF16) static_cast<uint16_t*>(dy_rep)[o] = static_cast<uint16_t>(pack_bf16x2(a, 0.f) & 0xFFFFu);
      else static_cast<float*>(dy_rep)[o] = a;
    }
    __syncthreads();
  }
}

// Gate gradients: one wave per token, a fixed-order float32 dot product per
// kept slot (0 for a dropped one).
template <bool BF16, int K>
__global__ __launch_bounds__(256) void cbwd_gate_kernel(const void* __restrict__ dy,
                                                        const void* __restrict__ y_rep,
                                                        const int32_t* __restrict__ rep_row,
                                                        const int32_t* __restrict__ slot_pos, int max_rows,
                                                        int T, int d, float* __restrict__ dgate) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  constexpr int EPC = BF16 ? 8 : 4;   // elements per 16-byte chunk
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * K + j];
    const int r = p >= 0 ? rep_row[p] : -1;
    float dot = 0.f;
    if (r >= 0 && r < max_rows) {
      for (int c = lane * EPC; c < d; c += 64 * EPC) {
        if constexpr (BF16) {
          const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(dy) +
                                                          static_cast<size_t>(t) * d + c);
          const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(y_rep) +
                                                          static_cast<size_t>(r) * d + c);
          const uint32_t uw[4] = {u.x, u.y, u.z, u.w}, vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            dot = fmaf(__uint_as_float(uw[i] << 16), __uint_as_float(vw[i] << 16), dot);
            dot = fmaf(__uint_as_float(uw[i] & 0xFFFF0000u), __uint_as_float(vw[i] & 0xFFFF0000u), dot);
          }
        } else {
          const float4 u = *reinterpret_cast<const float4*>(static_cast<const float*>(dy) +
                                                            static_cast<size_t>(t) * d + c);
          const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(y_rep) +
                                                            static_cast<size_t>(r) * d + c);
          dot = fmaf(u.x, v.x, dot);
          dot = fmaf(u.y, v.y, dot);
          dot = fmaf(u.z, v.z, dot);
          dot = fmaf(u.w, v.w, dot);
        }
      }
    }
    // fixed-order butterfly: every lane holds the same sum
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) dot += __shfl_xor(dot, o, 64);
    if (lane == 0) dgate[static_cast<size_t>(t) * K + j] = dot;
  }
}

}  // namespace
}  // namespace luffy

using namespace luffy;

extern "C" int luffy_combine(const void* y_rep, const int32_t* rep_row,
                             const int32_t* slot_pos, const float* topk_gate,
                             int T, int k, int d, int dtype, void* y, void* stream) {
  if (!y_rep || !rep_row || !slot_pos || !topk_gate || !y)
    return fail(LUFFY_E_INVALID, "luffy_combine: null pointer argument");
  if (T <= 0 || d <= 0) return fail(LUFFY_E_INVALID, "luffy_combine: T=%d d=%d", T, d);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "luffy_combine: k=%d must be 1 or 2", k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_combine: unknown dtype %d", dtype);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_combine: d=%d not a multiple of 64", d);
  if (static_cast<double>(T) * k * d * (dtype == LUFFY_BF16 ? 2 : 4) >= static_cast<double>(kRange))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_combine: y_rep of up to T*k=%lld rows of d=%d must span < 4 GiB - 64 KiB",
                static_cast<long long>(T) * k, d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int blocks = (T + 3) / 4;
  const bool two = d * (dtype == LUFFY_BF16 ? 2 : 4) <= 2 * 64 * 16;   // two chunks per lane cover a row
#define LUFFY_COMBINE(BF, K_, U_) launch("combine", combine_kernel<BF, K_, U_>, blocks, 256, 0, s, y_rep, rep_row, \
                                         slot_pos, topk_gate, T, d, y)
  if (dtype == LUFFY_BF16) {
    if (k == 1) { if (two) LUFFY_COMBINE(true, 1, 2); else LUFFY_COMBINE(true, 1, 4); }
    else { if (two) LUFFY_COMBINE(true, 2, 2); else LUFFY_COMBINE(true, 2, 4); }
  } else {
    if (k == 1) { if (two) LUFFY_COMBINE(false, 1, 2); else LUFFY_COMBINE(false, 1, 4); }
    else { if (two) LUFFY_COMBINE(false, 2, 2); else LUFFY_COMBINE(false, 2, 4); }
  }
#undef LUFFY_COMBINE
  return check_launch("luffy_combine");
}

extern "C" int luffy_combine_backward(const void* dy, const void* y_rep, const int32_t* rep_row,
                                      const int32_t* perm_token, const int32_t* slot_pos,
                                      const float* topk_gate, const int32_t* offsets,
                                      const int32_t* rep_offsets, int E, int T, int k, int d, int dtype,
                                      int max_rows, void* dy_rep, float* dgate, void* stream) {
  if (!dy || !y_rep || !rep_row || !perm_token || !slot_pos || !topk_gate || !offsets || !rep_offsets ||
      !dy_rep || !dgate)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: null pointer argument");
  if (T <= 0 || d <= 0 || E <= 0 || max_rows <= 0)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: T=%d d=%d E=%d max_rows=%d", T, d, E, max_rows);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "luffy_combine_backward: k=%d must be 1 or 2", k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: unknown dtype %d", dtype);
  if (E > 64) return fail(LUFFY_E_UNSUPPORTED, "luffy_combine_backward: E=%d > 64", E);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_combine_backward: d=%d not a multiple of 64", d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // work items: (representative ranges) x (d / 64); bounded by (max_rows / R + E) x (d / 64)
  const long long items = (static_cast<long long>(max_rows) / kGatherReps + E) * (d / kGatherCols);
  const int rows_blocks = static_cast<int>(std::min<long long>(items, 2048));
  const int blocks = (T + 3) / 4;
#define LUFFY_CBWD(BF, K_)                                                                                   \
  do {                                                                                                       \
    launch("cbwd_rows", cbwd_rows_kernel<BF, K_>, rows_blocks, 256, 0, s, dy, rep_row, perm_token, slot_pos, \
           topk_gate, offsets, rep_offsets, E, d, max_rows, dy_rep);                                         \
    launch("cbwd_gate", cbwd_gate_kernel<BF, K_>, blocks, 256, 0, s, dy, y_rep, rep_row, slot_pos, max_rows, \
           T, d, dgate);                                                                                     \
  } while (0)
  if (dtype == LUFFY_BF16) { if (k == 1) LUFFY_CBWD(true, 1); else LUFFY_CBWD(true, 2); }
  else { if (k == 1) LUFFY_CBWD(false, 1); else LUFFY_CBWD(false, 2); }
#undef LUFFY_CBWD
  return check_launch("luffy_combine_backward");
}

