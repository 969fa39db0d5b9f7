// Output tile of C[i][j] = sum_k P[i][k] * Q[j][k] on bf16 MFMA (gfx950).
//
// Both operands are row-major with the contraction index contiguous, so one
// core serves the similarity tiles (P and Q are gathered token rows of one
// bucket) and the FFN tiles (P = weight rows in [out, in] layout, Q =
// gathered token rows).  Operands go from global memory straight into LDS
// with buffer loads (buffer_load_dwordx4 ... lds, no staging registers;
// 32-bit byte offsets from a buffer resource, so each operand must span
// less than 4 GiB).  Operand rows are given as 32-bit element offsets from
// a base pointer (every operand here has fewer than 2^31 elements).  Waves
// are dealt to the four SIMDs of a CU round-robin (wave w on SIMD w % 4).
#pragma once

#include <type_traits>

#include "luffy_common.h"

namespace luffy {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 32 fp8 (OCP E4M3) values a lane: one operand fragment of the 32 x 32 x 64
// fp8 product.
typedef int i32x8 __attribute__((ext_vector_type(8)));

// v_mfma_scale_f32_32x32x64_f8f6f4 with both operands E4M3 (format 0) and
// unit block scales (E8M0 exponent 127 = 2^0).
__device__ __forceinline__ f32x16 mfma32x32x64_f8(i32x8 a, i32x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

// Workgroup barrier without the memory fences of __syncthreads(): the fence
// would make the compiler wait for every outstanding DMA load.  LDS
// visibility is handled explicitly: each wave waits (vmcnt) for its own DMA
// writes before the barrier, and LDS reads are issued after it.
__device__ __forceinline__ void raw_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with only the vector-memory counter constrained (<= N, N < 64;
// the 6-bit count is split over bits 3:0 and 15:14).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// threadIdx.x behind an empty volatile asm: values derived from it are
// recomputed where they are used instead of being hoisted out of a
// persistent kernel's tile loop, where they would stay live (and spill)
// across every tile shape the loop dispatches to.
__device__ __forceinline__ int opaque_tid() {
  int v = static_cast<int>(threadIdx.x);
  asm volatile("" : "+v"(v));
  return v;
}

// Tile core: output tile BM (P rows) x BN (Q rows), waves in a WM x WN
// grid, v_mfma_f32_32x32x16_bf16 blocks.  K advances BK (32 or 64) per
// stage through a ring of STAGES LDS stages; while one stage is multiplied
// the DMA of the next STAGES-1 is in flight.  Each operand row contributes
// BK*2 contiguous bytes per stage (a whole 128-byte line at BK = 64, which
// streams L2-resident operands at about twice the rate of 64-byte pieces;
// BK = 32 halves the stage and so allows a deeper ring, for operands that
// stream from HBM).  A DMA instruction fills 1 KB: 1024/(2*BK) rows.
// The 16-byte chunks of row r are stored XOR-permuted (BK = 64: by
// (r >> 1) & 7 over 8 chunks; BK = 32: by (r >> 2) & 3 over 4 chunks), so
// the 16 lanes of a fragment read (16 consecutive rows, one chunk) hit 16
// distinct bank groups.  K must be a multiple of BK.
//
// Wave placement: MFAST puts the P-block index fastest (wm = w % WM), so
// with WM = 4 each SIMD holds one P quarter of every Q part; QIL
// interleaves the Q blocks of the waves (wave wn owns 32-row Q blocks wn,
// wn + WN, ...).  In both cases a tile whose Q rows are only partly valid
// can skip the MFMAs of its invalid Q blocks (run<NQ>).
//
// Result layout of acc[fm][fn][v] in lane l of wave w:
//   P row  wave_m(w) * WTM + 32*fm + 8*(v/4) + 4*(l/32) + v%4
//   Q row  q_row(wave_n(w), fn) + l%32
//
// F8: the operands are fp8 (E4M3) rows, handed to the core as rows of
// 16-bit units (two values a unit: offsets, K and BK count units), so the
// DMA is unchanged; a 64-unit stage holds 128 values of K, multiplied in
// two steps of v_mfma_scale_f32_32x32x64_f8f6f4, whose fragments are two
// 16-byte chunks of a row (lanes 0-31 chunks 4s and 4s+1 of step s, lanes
// 32-63 chunks 4s+2 and 4s+3).  The accumulator layout is the same.
template <int BM_, int BN_, int WM_, int WN_, bool MFAST_, bool QIL_, int BK_ = 64, int STAGES_ = 2,
          bool PT_ = false, bool QT_ = false, bool F8_ = false>
struct GemmCore {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr bool QIL = QIL_;
  // K-major operands (PT: P, QT: Q): the operand is stored with its rows
  // along K (element (k, m) at k * ld + m), as a weight read transposed or
  // the token rows of a product that contracts over tokens.  Its stage holds
  // BK rows of k, each with the tile's BM (BN) values of m in 16-byte slots
  // XOR-permuted by swz_t(k); MFMA fragments are read with the transposing
  // LDS read (ds_read_b64_tr_b16), two per fragment.
  static constexpr bool PT = PT_, QT = QT_;
  static constexpr int BK = BK_;                     // K per stage
  static constexpr int STAGES = STAGES_;
  static_assert(BK == 32 || BK == 64, "stage width");
  static_assert(STAGES >= 2 && STAGES <= 5, "ring depth");
  static constexpr int THREADS = 64 * WM * WN;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 32, FN = WTN / 32;
  static constexpr int ROW_BYTES = BK * 2;
  static constexpr int CPR = ROW_BYTES / 16;         // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;               // rows per DMA instruction
  static constexpr bool F8 = F8_;
  static_assert(!F8 || (BK == 64 && !PT && !QT), "fp8 operands: row-major, 64-unit stages");
  static constexpr int STEPS = F8 ? BK / 32 : BK / 16;   // MFMA K steps per stage
  static constexpr int READS = F8 ? 2 : 1;               // LDS reads per fragment
  static constexpr int STAGE_BYTES = (BM + BN) * ROW_BYTES;
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
  static constexpr int NWAVES = WM * WN;
  // DMA instructions per wave and stage: LP of them P rows, LQ Q rows
  static constexpr int LP = BM / RPI / NWAVES, LQ = BN / RPI / NWAVES;
  static constexpr int LOADS = LP + LQ;
  static_assert(LP * NWAVES * RPI == BM && LQ * NWAVES * RPI == BN, "load plan");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  static_assert((STAGES - 1) * LOADS < 64, "vmcnt range");
  static constexpr int SLOTS_P = BM / 8, SLOTS_Q = BN / 8;   // 16-byte slots per k row (K-major)
  static_assert(!PT || (BK == 64 && (SLOTS_P == 16 || SLOTS_P == 32 || SLOTS_P == 64)), "K-major P tile");
  static_assert(!QT || (BK == 64 && (SLOTS_Q == 16 || SLOTS_Q == 32 || SLOTS_Q == 64)), "K-major Q tile");

  using Acc = f32x16[FM][FN];
  using lds_ptr = __attribute__((address_space(3))) uint8_t*;

  static __device__ __forceinline__ int swz(int r) { return BK == 64 ? (r >> 1) & 7 : (r >> 2) & 3; }
  // slot permutation of k row k of a K-major operand: the four k rows one
  // transposing read touches land on different slots
  static __device__ __forceinline__ int swz_t(int k) { return 2 * (k & 7); }
  static __device__ __forceinline__ int wave_m(int w) { return MFAST_ ? w % WM : w / WN; }
  static __device__ __forceinline__ int wave_n(int w) { return MFAST_ ? w / WM : w % WN; }
  static __device__ __forceinline__ int wave() { return __builtin_amdgcn_readfirstlane(opaque_tid() >> 6); }
  // first Q row of Q block fn of wave-column wn, and the row step between blocks
  static constexpr int QSTEP = QIL_ ? 32 * WN : 32;
  static __device__ __forceinline__ int q_row(int wn, int fn) { return (QIL_ ? 32 * wn : wn * WTN) + QSTEP * fn; }
  // Q blocks of wave-column wn that hold a valid row when rows are valid
  static __device__ __forceinline__ int active_q(int wn, int rows) {
    const int first = QIL_ ? 32 * wn : wn * WTN;
    return min(max((rows - first + QSTEP - 1) / QSTEP, 0), FN);
  }

  // Stage row this lane fills in load j: P rows 0..BM-1 (j < LP), then Q rows.
  static __device__ __forceinline__ int load_row(int j) {
    const int w = wave(), lane = opaque_tid() & 63;
    return (w + NWAVES * j) * RPI + lane / CPR;
  }

  // K-major operand, load j (P: j < LP, Q: j >= LP): the k row (0..BK-1) this
  // lane fills, and the element offset, at k = 0, of the 8 values it
  // fetches: k_row * ld + m_first + 8 * (slot ^ swz_t(k_row)); 0xFFFFFFFF
  // when those columns are at or past m_valid (not fetched).
  static __device__ __forceinline__ int kmajor_row(int j) {
    const int w = wave(), lane = opaque_tid() & 63;
    const bool isp = j < LP;
    const int slots = isp ? SLOTS_P : SLOTS_Q;
    return (w + NWAVES * (isp ? j : j - LP)) * (64 / slots) + lane / slots;
  }
  static __device__ __forceinline__ uint32_t kmajor_offset(int j, int ld, int m_first, int m_valid) {
    const int lane = opaque_tid() & 63;
    const int slots = j < LP ? SLOTS_P : SLOTS_Q;
    const int kr = kmajor_row(j);
    const int m = 8 * ((lane % slots) ^ swz_t(kr));
    return m < m_valid ? static_cast<uint32_t>(kr) * ld + m_first + m : 0xFFFFFFFFu;
  }

  static __device__ __forceinline__ void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }

  // Raw buffer resource over [base, base + kRange).  A row whose offset is
  // set to kRange is out of range: its buffer loads fetch nothing from
  // memory (robust buffer access), which is how rows past the valid ones
  // of a partial tile are skipped.  Valid rows need offset + K*2 <= kRange
  // (operands below 4 GiB - 64 KiB, K <= 32768).
  // The base is read from the first lane (it is wave-uniform by contract),
  // so the resource lives in scalar registers even when the compiler cannot
  // prove uniformity; a resource in vector registers would wrap every DMA
  // instruction in a readfirstlane loop.
  static constexpr uint32_t kRange = 0xFFFF0000u;
  static __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base) {
    const uint64_t v = reinterpret_cast<uint64_t>(base);
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v)));
    const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32)));
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>((hi << 32) | lo), static_cast<short>(0),
                                             static_cast<int>(kRange), 0x00020000);
  }

  // Stage kt: a row-major operand advances by the scalar offset kt*BK*2; a
  // K-major one by kt*BK rows of ld elements in its per-lane offset, and its
  // rows at or past kvalid are not fetched (they read as zeros).
  static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t prs, __amdgpu_buffer_rsrc_t qrs,
                                               const uint32_t (&goff)[LOADS], int kt, lds_ptr st, int w,
                                               int pld = 0, int qld = 0, int kvalid = 0x7fffffff) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      lds_ptr dst = st + (w + NWAVES * j) * 1024;
      const bool kmaj = j < LP ? PT : QT;
      uint32_t off = goff[j];
      int soff = kt * BK * 2;
      if (kmaj) {
        const int ld = j < LP ? pld : qld;
        const bool ok = off != kRange && kt * BK + kmajor_row(j) < kvalid;
        off = ok ? off + static_cast<uint32_t>(kt * BK) * static_cast<uint32_t>(ld) * 2u : kRange;
        soff = 0;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(j < LP ? prs : qrs,
                                               reinterpret_cast<__attribute__((address_space(3))) void*>(dst),
                                               16, off, soff, 0, 0);
    }
  }

  // lane fills physical chunk lane%CPR of its row with logical chunk
  // (lane%CPR) ^ swz(row); byte offsets.  P rows from pvalid on and Q rows
  // from qvalid on are marked out of range (not fetched).
  static __device__ __forceinline__ void dma_offsets(const uint32_t (&poff)[LP], const uint32_t (&qoff)[LQ],
                                                     int pvalid, int qvalid, uint32_t (&goff)[LOADS]) {
    const int lane = opaque_tid() & 63;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      if (j < LP ? PT : QT) {
        // K-major: the caller's kmajor_offset already places the 8 values
        const uint32_t o = j < LP ? poff[j] : qoff[j - LP];
        goff[j] = o == 0xFFFFFFFFu ? kRange : o * 2u;
        continue;
      }
      const int r = load_row(j);
      const uint32_t lc = static_cast<uint32_t>((lane % CPR) ^ swz(r));
      const bool valid = j < LP ? r < pvalid : r - BM < qvalid;
      goff[j] = valid ? ((j < LP ? poff[j] : qoff[j - LP]) + lc * 8) * 2u : kRange;
    }
  }

  // Fragments of one 16-wide K step (chunks 2*step and 2*step+1 of every
  // row: lanes 0-31 take the low chunk, lanes 32-63 the high one).
  using Frag = std::conditional_t<F8, i32x8, bf16x8>;
  struct Frags {
    Frag a[FM], b[FN];
  };

  // fp8 fragment: chunks c and c + 1 (byte offsets o0, o1) of a stage row
  static __device__ __forceinline__ i32x8 read_f8(lds_ptr row, int o0, int o1) {
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    const i32x4 lo = *reinterpret_cast<const __attribute__((address_space(3))) i32x4*>(row + o0);
    const i32x4 hi = *reinterpret_cast<const __attribute__((address_space(3))) i32x4*>(row + o1);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }

  // K step `step` of the stage at S, first NQ Q blocks.
  // One fragment of a K-major operand whose stage region starts at R (row
  // pitch PITCH bytes): lane l (group g = l/16, c = l%16) gets m = m_blk +
  // 16*(g%2) + c and k = 16*step + 8*(g/2) + 0..7, as the row-major read
  // does.  In each 16-lane group the transposing read hands lane c the
  // values (k0 + 0..3, m0 + c) when lane c addresses (k0 + c/4, m0 + 4*(c%4)).
  template <int PITCH>
  static __device__ __forceinline__ bf16x8 read_kmajor(lds_ptr R, int m_blk, int step) {
    typedef short v4i16 __attribute__((ext_vector_type(4)));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const int lane = opaque_tid() & 63;
    const int g = lane >> 4, c = lane & 15;
    const int m = m_blk + 16 * (g & 1) + 4 * (c & 3);
    const int k0 = 16 * step + 8 * (g >> 1) + (c >> 2);
    v4i16 h[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = k0 + 4 * u;
      lds_ptr a = R + k * PITCH + 16 * ((m >> 3) ^ swz_t(k)) + 2 * (m & 7);
      h[u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<__attribute__((address_space(3))) v4i16*>(a));
    }
    const v8i16 v = __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
  }

  template <int NQ>
  static __device__ __forceinline__ void read_step(lds_ptr S, int prow0, int qrow0, int half, int sw, int step,
                                                   Frags& f) {
    if constexpr (NQ > 0 && F8) {
      const int c0 = 4 * step + 2 * half;
      const int o0 = (c0 ^ sw) * 16, o1 = ((c0 + 1) ^ sw) * 16;
#pragma unroll
      for (int i = 0; i < FM; ++i) f.a[i] = read_f8(S + prow0 + 32 * i * ROW_BYTES, o0, o1);
#pragma unroll
      for (int j = 0; j < NQ; ++j) f.b[j] = read_f8(S + qrow0 + QSTEP * j * ROW_BYTES, o0, o1);
    } else if constexpr (NQ > 0) {
      const int pc = ((2 * step + half) ^ sw) * 16;
      if constexpr (PT) {
        const int wm = wave_m(wave());
#pragma unroll
        for (int i = 0; i < FM; ++i) f.a[i] = read_kmajor<BM * 2>(S, wm * WTM + 32 * i, step);
      } else {
#pragma unroll
        for (int i = 0; i < FM; ++i)
          f.a[i] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(S + prow0 +
                                                                                        32 * i * ROW_BYTES + pc);
      }
      if constexpr (QT) {
        const int wn = wave_n(wave());
#pragma unroll
        for (int j = 0; j < NQ; ++j) f.b[j] = read_kmajor<BN * 2>(S + BM * ROW_BYTES, q_row(wn, j), step);
      } else {
#pragma unroll
        for (int j = 0; j < NQ; ++j)
          f.b[j] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(S + qrow0 +
                                                                                        QSTEP * j * ROW_BYTES + pc);
      }
    }
  }

  template <int NQ>
  static __device__ __forceinline__ void mma_step(const Frags& f, Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < NQ; ++j) {
        if constexpr (F8) acc[i][j] = mfma32x32x64_f8(f.a[i], f.b[j], acc[i][j]);
        else acc[i][j] = mfma32x32x16(f.a[i], f.b[j], acc[i][j]);
      }
  }

  // Schedule of a step without buffer loads: the LDS reads of the next step
  // go out two per MFMA from the first MFMA on, so they have landed when the
  // next step starts.
  template <int NQ>
  static __device__ __forceinline__ void interleave_reads() {
    constexpr int NMF = FM * NQ, NDS = NQ > 0 ? READS * (FM + NQ) : 0;
#pragma unroll
    for (int i = 0; i < NMF; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      if (2 * i + 1 < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // DS read
      else if (2 * i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (NDS > 2 * NMF) __builtin_amdgcn_sched_group_barrier(0x100, NDS - 2 * NMF, 0);
  }

  // Schedule of the step after the barrier: the buffer loads of the next
  // stage to fetch go out first (one per MFMA), then the LDS reads; their
  // latency is the longer one.
  template <int NQ>
  static __device__ __forceinline__ void interleave_loads() {
    constexpr int NMF = FM * NQ, NDS = NQ > 0 ? READS * (FM + NQ) : 0, NVM = LOADS;
    constexpr int PV = NMF < NVM ? NMF : NVM;
    constexpr int PD = (NMF - PV) < NDS ? (NMF - PV) : NDS;
#pragma unroll
    for (int i = 0; i < PV; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
    }
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (NMF > PV + PD) __builtin_amdgcn_sched_group_barrier(0x008, NMF - PV - PD, 0);
    if constexpr (NVM > PV) __builtin_amdgcn_sched_group_barrier(0x020, NVM - PV, 0);
    if constexpr (NDS > PD) __builtin_amdgcn_sched_group_barrier(0x100, NDS - PD, 0);
  }

  // Wait until at most n stages of this wave's DMA are outstanding
  // (0 <= n <= STAGES - 2, wave-uniform).
  static __device__ __forceinline__ void wait_stages(int n) {
    if constexpr (STAGES > 4) {
      if (n >= 3) { wait_vmcnt<3 * LOADS>(); return; }
    }
    if constexpr (STAGES > 3) {
      if (n >= 2) { wait_vmcnt<2 * LOADS>(); return; }
    }
    if (n >= 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
  }

  // Steps ST..STEPS-1 of a stage (no buffer loads): step s reads step s of
  // the stage at S into f[s & 1] while multiplying f[(s - 1) & 1].
  template <int NQ, int ST>
  static __device__ __forceinline__ void inner_steps(lds_ptr S, int prow0, int qrow0, int half, int sw,
                                                     Frags (&f)[2], Acc& acc, bool sched) {
    if constexpr (ST < STEPS) {
      if (sched) __builtin_amdgcn_sched_barrier(0);
      read_step<NQ>(S, prow0, qrow0, half, sw, ST, f[ST & 1]);
      mma_step<NQ>(f[(ST - 1) & 1], acc);
      if (sched) interleave_reads<NQ>();
      inner_steps<NQ, ST + 1>(S, prow0, qrow0, half, sw, f, acc, sched);
    }
  }

  // DMA state of a tile between prefetch() and resume().
  struct Pipe {
    __amdgpu_buffer_rsrc_t prs, qrs;
    uint32_t goff[LOADS];
    int nk, pld, qld, kvalid;
  };

  // First half of run(): issues the DMA of the tile's first min(K/BK,
  // STAGES) stages into the LDS ring (every stage buffer must be free: after
  // a run()/resume() of the previous tile, whose closing barrier
  // guarantees it).  A persistent kernel calls it before the previous
  // tile's epilogue so that the epilogue hides the fetch latency; the
  // epilogue must then keep out of the ring's LDS.
  static __device__ __forceinline__ void prefetch(const uint16_t* __restrict__ pbase, const uint32_t (&poff)[LP],
                                                  const uint16_t* __restrict__ qbase, const uint32_t (&qoff)[LQ],
                                                  int K, int pvalid, int qvalid, uint8_t* lds_generic, Pipe& p,
                                                  int pld = 0, int qld = 0, int kvalid = 0x7fffffff) {
    const lds_ptr lds = (lds_ptr)lds_generic;
    const int w = wave();
    p.prs = rsrc(pbase);
    p.qrs = rsrc(qbase);
    p.pld = pld;
    p.qld = qld;
    p.kvalid = kvalid;
    dma_offsets(poff, qoff, pvalid, qvalid, p.goff);
    p.nk = __builtin_amdgcn_readfirstlane(K / BK);
    const int pro = min(p.nk, STAGES);
#pragma unroll
    for (int s = 0; s < STAGES; ++s)
      if (s < pro) issue(p.prs, p.qrs, p.goff, s, lds + s * STAGE_BYTES, w, pld, qld, kvalid);
  }

  // poff[j] (j < LP): element offset of P row load_row(j);
  // qoff[j] (j < LQ): element offset of Q row load_row(LP + j) - BM.
  // Only the first pvalid P rows and qvalid Q rows are fetched; the LDS
  // rows of the others hold stale values, which only reach accumulator rows
  // and columns of invalid rows.  Ends with a barrier after which the LDS
  // may be reused.  NQ: the wave multiplies only its first NQ Q blocks;
  // every wave still issues its share of the loads and takes every barrier.
  //
  // Fragments are double-buffered per 16-wide K step: while the MFMAs of
  // step s run, the fragments of step s+1 are read.  Stage kt (buffer
  // kt % STAGES): steps 1..STEPS-1 are read while steps 0..STEPS-2 are
  // multiplied; then wait for stage kt+1 and for this wave's reads, barrier
  // (every wave is done with buffer kt % STAGES), issue the DMA of stage
  // kt+STAGES into it and read step 0 of stage kt+1 while the last step is
  // multiplied.  Holding one step per buffer keeps the FFN tile within 256
  // registers per lane without register reuse stalls.
  // pld, qld: row pitch (elements) of a K-major P / Q; kvalid: K rows of
  // K-major operands at or past it read as zeros (rows beyond an expert's).
  template <int NQ = FN>
  static __device__ __forceinline__ void run(const uint16_t* __restrict__ pbase, const uint32_t (&poff)[LP],
                                             const uint16_t* __restrict__ qbase, const uint32_t (&qoff)[LQ],
                                             int K, int pvalid, int qvalid, uint8_t* lds_generic, Acc& acc,
                                             int pld = 0, int qld = 0, int kvalid = 0x7fffffff) {
    Pipe p;
    prefetch(pbase, poff, qbase, qoff, K, pvalid, qvalid, lds_generic, p, pld, qld, kvalid);
    resume<NQ>(p, lds_generic, acc);
  }

  // fp8 step: the MFMAs of the fragments in f, while the fragments of step
  // `step` of the stage at S are read into f: the B fragments into a
  // second set first, then A fragment i as soon as the MFMAs that use it
  // are issued.  Two sets of 32-byte fragments would not fit beside the
  // accumulators.  READ = false: the MFMAs only.
  // NV: DMA instructions issued just before (the stage after the barrier),
  // spread one after each MFMA.
  template <int NQ, bool READ, int NV = 0>
  static __device__ __forceinline__ void mma_read_f8(lds_ptr S, int prow0, int qrow0, int half, int sw, int step,
                                                     Frags& f, Acc& acc) {
    const int c0 = 4 * step + 2 * half;
    const int o0 = (c0 ^ sw) * 16, o1 = ((c0 + 1) ^ sw) * 16;
    Frag nb[NQ > 0 ? NQ : 1];
    if constexpr (READ) {
#pragma unroll
      for (int j = 0; j < NQ; ++j) nb[j] = read_f8(S + qrow0 + QSTEP * j * ROW_BYTES, o0, o1);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < NQ; ++j) acc[i][j] = mfma32x32x64_f8(f.a[i], f.b[j], acc[i][j]);
      if constexpr (READ) f.a[i] = read_f8(S + prow0 + 32 * i * ROW_BYTES, o0, o1);
    }
    if constexpr (READ) {
#pragma unroll
      for (int j = 0; j < NQ; ++j) f.b[j] = nb[j];
      // MFMAs of A fragment i (each followed by one DMA while any is left),
      // then its next-step reads, then one B fragment of the next step
#pragma unroll
      for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if (i * NQ + j < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        if (i < NQ) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      constexpr int REST = NV > FM * NQ ? NV - FM * NQ : 0;
      if constexpr (REST > 0) __builtin_amdgcn_sched_group_barrier(0x020, REST, 0);
    }
  }

  // resume() for fp8 operands: the same ring and barriers, one fragment set.
  template <int NQ>
  static __device__ __forceinline__ void resume_f8(const Pipe& p, uint8_t* lds_generic, Acc& acc) {
    const lds_ptr lds = (lds_ptr)lds_generic;
    const int lane = opaque_tid() & 63;
    const int w = wave();
    const int wm = wave_m(w), wn = wave_n(w);
    const __amdgpu_buffer_rsrc_t prs = p.prs, qrs = p.qrs;
    uint32_t goff[LOADS];
#pragma unroll
    for (int j = 0; j < LOADS; ++j) goff[j] = p.goff[j];
    const int nk = p.nk;
    const int pro = min(nk, STAGES);
    wait_stages(pro - 1);
    raw_barrier();
    const int sw = swz(lane & 31);
    const int prow0 = (wm * WTM + (lane & 31)) * ROW_BYTES;
    const int qrow0 = (BM + q_row(wn, 0) + (lane & 31)) * ROW_BYTES;
    const int half = lane >> 5;
    Frags f;
    read_step<NQ>(lds, prow0, qrow0, half, sw, 0, f);
    int kt = 0, cb = 0;
    // steady state: stage kt+STAGES exists
    for (; kt + STAGES < nk; ++kt) {
      const lds_ptr cur = lds + cb * STAGE_BYTES;
      cb = cb + 1 == STAGES ? 0 : cb + 1;
      const lds_ptr nxt = lds + cb * STAGE_BYTES;
#pragma unroll
      for (int st = 1; st < STEPS; ++st) {
        __builtin_amdgcn_sched_barrier(0);
        mma_read_f8<NQ, true>(cur, prow0, qrow0, half, sw, st, f, acc);
      }
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<(STAGES - 2) * LOADS>();   // stage kt+1 landed (this wave's part)
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): own reads of stage kt done
      raw_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue(prs, qrs, goff, kt + STAGES, cur, w);
      mma_read_f8<NQ, true, LOADS>(nxt, prow0, qrow0, half, sw, 0, f, acc);
      __builtin_amdgcn_sched_barrier(0);
    }
    // last stages: nothing more to issue; the reads that follow the very
    // last step fetch unused values from a stage that is still intact
    for (; kt < nk; ++kt) {
      const lds_ptr cur = lds + cb * STAGE_BYTES;
      cb = cb + 1 == STAGES ? 0 : cb + 1;
#pragma unroll
      for (int st = 1; st < STEPS; ++st) mma_read_f8<NQ, true>(cur, prow0, qrow0, half, sw, st, f, acc);
      const bool more = kt + 1 < nk;
      if (more) {
        wait_stages(nk - 2 - kt);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        raw_barrier();
      }
      mma_read_f8<NQ, true>(more ? lds + cb * STAGE_BYTES : cur, prow0, qrow0, half, sw, 0, f, acc);
    }
    __syncthreads();
  }

  // Second half of run(): waits for the prefetched stages and runs the K
  // loop; ends with a barrier after which the LDS may be reused.
  template <int NQ = FN>
  static __device__ __forceinline__ void resume(const Pipe& p, uint8_t* lds_generic, Acc& acc) {
    if constexpr (F8) {
      resume_f8<NQ>(p, lds_generic, acc);
      return;
    }
    const lds_ptr lds = (lds_ptr)lds_generic;
    const int lane = opaque_tid() & 63;
    const int w = wave();
    const int wm = wave_m(w), wn = wave_n(w);
    const __amdgpu_buffer_rsrc_t prs = p.prs, qrs = p.qrs;
    const int pld = p.pld, qld = p.qld, kvalid = p.kvalid;
    uint32_t goff[LOADS];
#pragma unroll
    for (int j = 0; j < LOADS; ++j) goff[j] = p.goff[j];
    const int nk = p.nk;
    const int pro = min(nk, STAGES);
    wait_stages(pro - 1);
    raw_barrier();
    const int sw = swz(lane & 31);
    const int prow0 = (wm * WTM + (lane & 31)) * ROW_BYTES;
    const int qrow0 = (BM + q_row(wn, 0) + (lane & 31)) * ROW_BYTES;
    const int half = lane >> 5;
    Frags f[2];
    read_step<NQ>(lds, prow0, qrow0, half, sw, 0, f[0]);
    int kt = 0, cb = 0;   // stage and its buffer
    // steady state: stage kt+STAGES exists
    for (; kt + STAGES < nk; ++kt) {
      const lds_ptr cur = lds + cb * STAGE_BYTES;
      cb = cb + 1 == STAGES ? 0 : cb + 1;
      const lds_ptr nxt = lds + cb * STAGE_BYTES;
      inner_steps<NQ, 1>(cur, prow0, qrow0, half, sw, f, acc, true);
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<(STAGES - 2) * LOADS>();   // stage kt+1 landed (this wave's part)
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): own reads of stage kt done
      raw_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue(prs, qrs, goff, kt + STAGES, cur, w, pld, qld, kvalid);
      read_step<NQ>(nxt, prow0, qrow0, half, sw, 0, f[0]);
      mma_step<NQ>(f[1], acc);
      interleave_loads<NQ>();
      __builtin_amdgcn_sched_barrier(0);
    }
    // last stages: nothing more to issue
    for (; kt < nk; ++kt) {
      const lds_ptr cur = lds + cb * STAGE_BYTES;
      cb = cb + 1 == STAGES ? 0 : cb + 1;
      inner_steps<NQ, 1>(cur, prow0, qrow0, half, sw, f, acc, false);
      if (kt + 1 < nk) {
        wait_stages(nk - 2 - kt);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        raw_barrier();
        read_step<NQ>(lds + cb * STAGE_BYTES, prow0, qrow0, half, sw, 0, f[0]);
      }
      mma_step<NQ>(f[1], acc);
    }
    __syncthreads();
  }
};

// 256 x 256, 512 threads, wave tile 128 x 64, 64-wide stages.
using GemmBig64 = GemmCore<256, 256, 2, 4, false, false>;
// The same on fp8 rows: 128 values of K a stage.
using GemmBig64F8 = GemmCore<256, 256, 2, 4, false, false, 64, 2, false, false, true>;
// 256 x 256, 512 threads, wave tile 64 x 128 (SIMD s holds P rows
// 64s..64s+63 of both Q halves), 64-wide stages.
using GemmRagged64 = GemmCore<256, 256, 4, 2, true, false>;

// Persistent-kernel block order: consecutive virtual ids share an XCD
// (workgroups are dealt to the 8 XCDs round-robin), so the tiles that run
// together on one XCD are neighbours in tile order and share its L2.
__device__ __forceinline__ int xcd_virtual_block() {
  constexpr int kXcds = 8;
  const int g = gridDim.x, b = blockIdx.x;
  if (g % kXcds) return b;
  return (b % kXcds) * (g / kXcds) + b / kXcds;
}

// Work item of round r of a persistent block with virtual id vb: rounds
// alternate direction, so a block that drew one of the first items of a
// round draws one of the last of the next.  With tiles of two alternating
// kinds (a full and a partial token tile per weight tile) every block then
// gets one of each instead of two of the same.  Every item below total is
// visited exactly once.
__device__ __forceinline__ int serpentine_item(int round, int vb) {
  const int g = gridDim.x;
  return round * g + ((round & 1) ? g - 1 - vb : vb);
}

}  // namespace luffy
