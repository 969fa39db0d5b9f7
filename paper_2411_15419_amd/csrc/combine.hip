// luffy_combine: y[t] = sum over kept slots j of gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
// One wave per token; 16-byte vector loads and stores; float32 sums.
#include "luffy_common.h"

namespace luffy {
namespace {

template <bool BF16>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y_rep,
                                                      const int32_t* __restrict__ rep_row,
                                                      const int32_t* __restrict__ slot_pos,
                                                      const float* __restrict__ gate, int T, int k,
                                                      int d, void* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int row[2] = {-1, -1};
  float g[2] = {0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * k + j];
    if (p >= 0) {
      row[j] = rep_row[p];
      g[j] = gate[static_cast<size_t>(t) * k + j];
    }
  }
  if constexpr (BF16) {
    const uint16_t* src = static_cast<const uint16_t*>(y_rep);
    uint16_t* dst = static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d;
    for (int c = lane * 8; c < d; c += 512) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int j = 0; j < k; ++j) {
        if (row[j] < 0) continue;
        Pack16 v;
        v.u4 = *reinterpret_cast<const uint4*>(src + static_cast<size_t>(row[j]) * d + c);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(g[j], bf16_to_f32(v.h[i]), acc[i]);
      }
      Pack16 o;
#pragma unroll
      for (int i = 0; i < 8; ++i) o.h[i] = f32_to_bf16(acc[i]);
      *reinterpret_cast<uint4*>(dst + c) = o.u4;
    }
  } else {
    const float* src = static_cast<const float*>(y_rep);
    float* dst = static_cast<float*>(y) + static_cast<size_t>(t) * d;
    for (int c = lane * 4; c < d; c += 256) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int j = 0; j < k; ++j) {
        if (row[j] < 0) continue;
        const float4 v = *reinterpret_cast<const float4*>(src + static_cast<size_t>(row[j]) * d + c);
        acc.x = fmaf(g[j], v.x, acc.x);
        acc.y = fmaf(g[j], v.y, acc.y);
        acc.z = fmaf(g[j], v.z, acc.z);
        acc.w = fmaf(g[j], v.w, acc.w);
      }
      *reinterpret_cast<float4*>(dst + c) = acc;
    }
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int blocks = (T + 3) / 4;
  ProfileScope prof_("combine", s);
  if (dtype == LUFFY_BF16)
    combine_kernel<true><<<blocks, 256, 0, s>>>(y_rep, rep_row, slot_pos, topk_gate, T, k, d, y);
  else
    combine_kernel<false><<<blocks, 256, 0, s>>>(y_rep, rep_row, slot_pos, topk_gate, T, k, d, y);
  return check_launch("luffy_combine");
}
