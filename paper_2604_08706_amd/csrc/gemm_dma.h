// The K loop of every bf16 product: operands streamed HBM -> LDS with direct
// loads (gfx950 buffer_load_dwordx4 ... lds), K step 64, two LDS stages.
//
// * Direct loads need no staging registers and no ds_write instructions.  A
//   load instruction writes 64 lanes x 16 bytes to LDS at M0 + 16 * lane, i.e.
//   8 consecutive 128-byte rows; the bank swizzle (gemm_core.h) is applied on
//   the HBM side -- the lane that lands on physical chunk p of row `row`
//   fetches logical chunk p ^ swz(row).
// * 128-byte rows make every row segment a whole cache line: measured L2 ->
//   CU rate ~28 TB/s for 128-byte segments against ~16 TB/s for 64-byte ones.
// * The loads of step s + 1 are issued right after the barrier that frees
//   their stage -- one full step ahead -- half during the last K slice of one
//   step and half during the first slice of the next, spread between MFMAs so
//   the wave's MFMA issue never waits behind a burst of loads.
// * Fragments are read one K slice (16) ahead of the MFMAs that use them; the
//   first slice of step s + 1 is read right after the barrier, while the last
//   slice of step s (already in registers) multiplies.
// * The loads are issued with inline assembly and their completion is tracked
//   by hand (s_waitcnt vmcnt): the compiler's own tracking of LDS-DMA waits for
//   every outstanding load before each LDS read and would serialize the
//   pipeline.  Nothing else in these kernels touches M0 or issues vector memory
//   loads inside the loop, and the loop ends with vmcnt(0).
#pragma once

#include "gemm_core.h"

namespace rbp {
namespace gemm {

constexpr int kBK = 64;
constexpr int kStageBytes = 2 * kTileBytes;  // A + B
static_assert(2 * kStageBytes <= kLdsBytes, "two stages must fit the LDS allocation");

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource as four SGPRs: 48-bit base, stride 0, range in bytes.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from buffer offset `voff` into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, i32x4 rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt encodings (gfx9): vmcnt in bits [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]; other counters left at their maximum.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Workgroup barrier that is also a compiler memory barrier: LDS reads after it
// may not be moved above it (s_barrier alone orders no memory accesses).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <class G>
__device__ __forceinline__ void mfma_tiles(const bf16x8 (&a)[G::MI], const bf16x8 (&b)[G::NI],
                                           f32x16 (&acc)[G::MI][G::NI]) {
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
}

// MFMAs of one K slice with `nload` loads spread evenly between them: a
// burst of loads would stall this wave's MFMA issue while the CU's address
// unit accepts them.  load(l) issues load l (or nothing).
template <class G, class LoadFn>
__device__ __forceinline__ void mfma_tiles_interleaved(const bf16x8 (&a)[G::MI],
                                                       const bf16x8 (&b)[G::NI],
                                                       f32x16 (&acc)[G::MI][G::NI], int nload,
                                                       LoadFn&& load) {
  constexpr int M = G::MI * G::NI;
  const int every = M / nload;
#pragma unroll
  for (int q = 0; q < M; ++q) {
    const int mi = q / G::NI, ni = q % G::NI;
    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    if ((q + 1) % every == 0 && (q + 1) / every <= nload) {
      RBP_FENCE();
      load((q + 1) / every - 1);
      RBP_FENCE();
    }
  }
}

template <class G>
struct DmaOperand {
  static constexpr int kLoads = 32 / G::kWaves;  // 1 KiB blocks per wave per step
  i32x4 rsrc;
  uint32_t voff[kLoads];
  int kc[kLoads];
  int64_t k_extent;

  __device__ __forceinline__ void init(const Operand& op, int64_t mn0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t rows = op.mn_extent - mn0;
    rows = rows < 0 ? 0 : (rows > 256 ? 256 : rows);
    rsrc = rsrc_words(op.ptr + mn0 * op.ld, (uint32_t)(rows * op.ld * 2));
    // block b = j * kWaves + wave holds rows 8 b .. 8 b + 7; lane -> row
    // 8 b + lane / 8, physical chunk lane % 8, logical chunk
    // (lane % 8) ^ swz(row), swz(row) = (row ^ (row >> 3)) & 7 = (lane / 8) ^ (b & 7)
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int b = j * G::kWaves + wave;
      const int row = b * 8 + (lane >> 3);
      const int c = (lane & 7) ^ (lane >> 3) ^ (b & 7);
      kc[j] = c * 8;
      voff[j] = (uint32_t)((row * op.ld + c * 8) * 2);
    }
    k_extent = op.k_extent;
  }
  __device__ __forceinline__ void issue_one(uint32_t tile, int64_t k0, int j) const {
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool ok = k0 + kc[j] < k_extent;
    dma16(tile + (uint32_t)(j * G::kWaves + wave) * 1024u,
          ok ? voff[j] + (uint32_t)(k0 * 2) : kOutOfRange, rsrc);
  }
};

// Fragment bases for 128-byte rows (gemm_core.h swizzle): slice ks, row block i
// reads base[((2 ks) ^ (4 (i & 1))) / 2] + 4096 i.
struct FragBase {
  uint32_t a[4], b[4];
};

template <class G>
__device__ __forceinline__ FragBase frag_bases() {
  const int lane = threadIdx.x & 63;
  const int r = lane & 31;
  const int t = (lane >> 5) ^ (r & 7) ^ (r >> 3);
  FragBase f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t off = (uint32_t)(r * 128 + (((2 * j) ^ t) << 4));
    f.a[j] = (uint32_t)(G::wm() * (256 / G::WM) * 128) + off;
    f.b[j] = (uint32_t)(kTileBytes + G::wn() * (256 / G::WN) * 128) + off;
  }
  return f;
}

template <class G>
__device__ __forceinline__ void read_frags(const uint8_t* stage, const FragBase& f, int ks,
                                        bf16x8 (&a)[G::MI], bf16x8 (&b)[G::NI]) {
#pragma unroll
  for (int i = 0; i < G::MI; ++i)
    a[i] = *reinterpret_cast<const bf16x8*>(stage + f.a[((2 * ks) ^ (4 * (i & 1))) >> 1] +
                                            4096 * i);
#pragma unroll
  for (int i = 0; i < G::NI; ++i)
    b[i] = *reinterpret_cast<const bf16x8*>(stage + f.b[((2 * ks) ^ (4 * (i & 1))) >> 1] +
                                            4096 * i);
}

// Full K loop over [k_begin, k_end) for the tile at (m0, n0), both operands
// K-major (k_extent % 8 == 0), K step 64, two LDS stages.  Per step s (stage
// s % 2), with slice 0's fragments already in registers:
//   slices 0..2: read the next slice's fragments, then this slice's MFMAs
//     (slice 0 also issues step s + 1's B loads, deferred from step s - 1);
//   wait for step s + 1's loads and for this wave's LDS reads; barrier
//     (step s + 1 visible; stage s % 2 no longer read by anyone);
//   read step s + 1's slice 0 fragments; slice 3's MFMAs, issuing step s + 2's
//     A loads into stage s % 2.
// Ends with a barrier, so the caller may reuse `smem` right away.
template <class G>
__device__ __forceinline__ void mainloop(const Operand& A, const Operand& B, int64_t m0,
                                         int64_t n0, int64_t k_begin, int64_t k_end,
                                         uint8_t* smem, f32x16 (&acc)[G::MI][G::NI]) {
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
  const int64_t nk = (k_end - k_begin + kBK - 1) / kBK;
  if (nk <= 0) return;
  constexpr int L = DmaOperand<G>::kLoads;
  DmaOperand<G> la, lb;
  la.init(A, m0);
  lb.init(B, n0);
  const FragBase f = frag_bases<G>();
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);
  auto stage_lds = [&](int64_t step) { return lds0 + (uint32_t)(step & 1) * kStageBytes; };
  auto kof = [&](int64_t step) { return k_begin + step * kBK; };
  // prologue: step 0 landed, step 1 in flight
#pragma unroll
  for (int j = 0; j < L; ++j) la.issue_one(stage_lds(0), kof(0), j);
#pragma unroll
  for (int j = 0; j < L; ++j) lb.issue_one(stage_lds(0) + kTileBytes, kof(0), j);
  wait_vmcnt<0>();
  lds_barrier();
  if (nk > 1) {
#pragma unroll
    for (int j = 0; j < L; ++j) la.issue_one(stage_lds(1), kof(1), j);
#pragma unroll
    for (int j = 0; j < L; ++j) lb.issue_one(stage_lds(1) + kTileBytes, kof(1), j);
  }
  bf16x8 a0[G::MI], b0[G::NI], a1[G::MI], b1[G::NI];
  read_frags<G>(smem, f, 0, a0, b0);
  for (int64_t it = 0; it < nk; ++it) {
    const uint8_t* cur = smem + (it & 1) * kStageBytes;
    const uint8_t* nxt = smem + ((it + 1) & 1) * kStageBytes;
    // B loads of step it + 1, deferred from the previous step's last slice
    const bool b_due = it >= 1 && it + 1 < nk;
    const uint32_t st1 = stage_lds(it + 1) + kTileBytes;
    const int64_t k1 = kof(it + 1);
    read_frags<G>(cur, f, 1, a1, b1);
    RBP_FENCE();
    mfma_tiles_interleaved<G>(a0, b0, acc, L, [&](int l) {
      if (b_due) lb.issue_one(st1, k1, l);
    });
    RBP_FENCE();
    read_frags<G>(cur, f, 2, a0, b0);
    RBP_FENCE();
    mfma_tiles<G>(a1, b1, acc);
    RBP_FENCE();
    read_frags<G>(cur, f, 3, a1, b1);
    RBP_FENCE();
    mfma_tiles<G>(a0, b0, acc);
    RBP_FENCE();
    // step it + 1 landed (only its loads are outstanding); this wave's reads
    // of stage it % 2 done, so after the barrier the stage may be refilled
    __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) lgkmcnt(0)
    lds_barrier();
    // unconditional (the last step re-reads a stale stage): a read under a
    // branch would make the compiler wait for it before the MFMAs below
    read_frags<G>(nxt, f, 0, a0, b0);
    RBP_FENCE();
    const bool a_due = it + 2 < nk;
    const uint32_t st2 = stage_lds(it + 2);
    const int64_t k2 = kof(it + 2);
    mfma_tiles_interleaved<G>(a1, b1, acc, L, [&](int l) {
      if (a_due) la.issue_one(st2, k2, l);
    });
    RBP_FENCE();
  }
  wait_vmcnt<0>();
  __syncthreads();
}

}  // namespace gemm
}  // namespace rbp
