// luffy_combine: y[t] = sum over kept slots j of gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
// One wave per token; 16-byte vector loads and stores (four per lane in
// flight per source row, eight in all); float32 sums.
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
