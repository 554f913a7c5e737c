// kernels.hip -- gfx950 (MI355X, CDNA4) kernels of the MoE expert stage.
//
//  * producer: persistent rank-wide grouped GEMMs (paper Section 3.3.1), one
//    launch for the fused gate/up projection (an item = 256 rows x 128 ffn
//    features, both projections, SiLU-gated in the epilogue) and one for the
//    down projection (an item = 256 rows x 256 hidden columns).  A queue per
//    launch covers every local expert.  Each finished down tile of a tile row
//    that needs a transfer publishes a ready flag with an agent-scope release
//    (the epilogue signal of Section 3.3.1).
//  * consumer: persistent kernel on its own compute units (Section 3.3.3)
//    that polls the flags of whole segments (Section 3.3.2) and copies each
//    ready segment into its destination receive buffer.
//  * scatter: the non-overlapped baseline's bulk return copy.
//  * init: resets the per-run counters (a kernel, not a memset, so the
//    sequence stays capturable).
//
// Math: bf16 operands, v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  The
// weight tile is the MFMA A operand (output features on the MFMA M side) and
// the token tile is the B operand, so every lane ends up holding 4
// consecutive output features of one token row and stores 8 bytes at a time.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.hpp"

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Global-memory view of a pointer that was loaded from memory (the receive-buffer table): the
// compiler cannot infer its address space and would emit flat accesses.
typedef __attribute__((address_space(1))) u32x4 g_u32x4;

// Operand tiles in LDS: 256 rows x 32 k (bf16) = 16 KiB per operand, 64 bytes per row,
// weight tile then token tile per stage, four stages in a ring (128 KiB).  Global
// memory is copied straight into LDS with global_load_lds_dwordx4 (no register
// staging), three K-steps ahead of the MFMAs.  A DMA instruction writes 64 lanes x 16
// bytes contiguously, i.e. 16 rows, so each lane fetches the 16-byte chunk that
// belongs at its slot: chunk c of row r sits at physical chunk c ^ g(r).  g spreads the
// 32 rows that one MFMA operand read touches over all banks, for 8-lane (32-bank) and
// 16-lane (64-bank) phases alike.
constexpr int kRowBytes = kTileK * 2;                  // 64
constexpr int kOperandBytes = kTileM * kRowBytes;      // 16 KiB
constexpr int kStageBytes = 2 * kOperandBytes;         // 32 KiB
constexpr int kStages = 4;
constexpr int kLdsBytes = kStages * kStageBytes;       // 128 KiB (operand ring)
constexpr int kRowsPerDma = 64 * 16 / kRowBytes;       // 16 rows per DMA instruction
// Epilogue staging: the finished tile goes through LDS (free once the pipeline drains) so
// that global stores are whole 16-byte chunks of contiguous rows.  Rows are padded by 16
// bytes so the 32 lanes writing one column of 32 rows hit distinct banks.
constexpr int kDownOutStride = kDownTileN * 2 + 16;    // 528 B per staged output row
constexpr int kGuOutStride = kGuTileF * 2 + 16;        // 272 B per staged activation row
constexpr int kLdsAlloc = kTileM * kDownOutStride;     // 135168 B >= the 128 KiB operand ring
constexpr int kDmaPerThread = kTileM / kRowsPerDma / 4;  // 4 per operand per thread

// Chunk swizzle of the 64-byte operand rows: a row's four 16-byte K chunks are stored XOR
// ((row / 2) ^ (row / 8)) % 4.  Measured on gfx950, fragment reads with it spend half of their
// LDS-active cycles on bank conflicts, and (row / 4) % 4 brings that to 2 %; but the latter
// costs the gate/up kernel a vector register, pushing it past the budget that lets two
// consumer waves share its SIMDs, and the stage time did not change measurably.
__device__ __forceinline__ uint32_t swz(uint32_t row) { return ((row >> 1) ^ (row >> 3)) & 3u; }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

__device__ __forceinline__ uint64_t ticks() { return wall_clock64(); }

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)LDS_PTR(p);
}

// 16 bytes per lane from global memory (scalar base + 32-bit lane offset) straight into
// LDS at M0 + 16 * lane.  Issued as inline assembly so that the compiler's wait-count
// pass does not serialise LDS reads behind every in-flight DMA: the pipeline waits for
// exactly the stage it needs with an explicit vmcnt.  M0 is written right before the
// load and is not used by any compiler-generated code in the producer.
// 8 bytes stored as a relaxed agent-scope atomic store: it completes at the device's coherence
// point, so once every wave's stores have completed (an explicit vmcnt(0) before a barrier)
// another XCD can read the data after an agent-scope acquire, and the writer needs no L2
// writeback to publish it.  A relaxed flag store or arrival count then follows.  Callers lay
// data out so that the 64 lanes of a wave store 512 contiguous bytes (whole cache lines).
__device__ __forceinline__ void store8_device(void* p, uint64_t v) {
  __hip_atomic_store((uint64_t*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t pack_f32x2(float lo, float hi) {
  return (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32);
}

__device__ __forceinline__ void dma16(const uint8_t* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(sbase)
               : "memory");
}

// Waits until at most n of this wave's global loads are outstanding and all LDS reads have
// returned, then joins the workgroup barrier.  The empty asm statements keep the compiler
// from moving memory operations across the barrier; no fence is emitted, so in-flight
// LDS-DMA loads of later stages stay in flight.
template <int n>
__device__ __forceinline__ void wait_vm_and_barrier() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  // gfx9 s_waitcnt: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14, expcnt 6:4, lgkmcnt 11:8.
  constexpr int imm = (n & 15) | ((n >> 4) << 14) | (7 << 4) | (0 << 8);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(imm);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------------------
// One 256x256 output tile: acc[i][j] holds D[n][m] for the wave's 128x128
// quadrant, n = wn*128 + i*32 + 8*(r/4) + 4*(lane/32) + r%4, m = wm*128 + j*32 + lane%32.
// wbase / xbase are wave-uniform byte bases of the weight / token operand; woff[i] /
// xoff[i] are this lane's byte offsets of the row it fetches for DMA instruction i
// (operand-tile row (wave*4 + i)*16 + lane/4), including its swizzled 16-byte chunk.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void tile_mma(uint8_t* __restrict__ lds, const uint8_t* wbase, const uint8_t* xbase,
                                         const uint32_t (&woff)[kDmaPerThread],
                                         const uint32_t (&xoff)[kDmaPerThread], int K, f32x16 (&acc)[4][4]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave & 1, wm = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;
  const uint32_t lsw = swz(lr);
  const uint32_t a_row = (uint32_t)(wn * 128 + lr) * kRowBytes;
  const uint32_t b_row = (uint32_t)(wm * 128 + lr) * kRowBytes;
  const uint32_t dma_off = (uint32_t)wave * kDmaPerThread * 1024;

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  const int nk = K / kTileK;
  const uint32_t lds0 = lds_addr(lds) + dma_off;
  auto issue = [&](int ks) {
    const uint32_t st = lds0 + (uint32_t)(ks & (kStages - 1)) * kStageBytes;
    const uint8_t* wb = wbase + ks * kRowBytes;  // wave-uniform: scalar base + 32-bit lane offset
    const uint8_t* xb = xbase + ks * kRowBytes;
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) dma16(wb, woff[i], st + i * 1024);
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) dma16(xb, xoff[i], st + kOperandBytes + i * 1024);
  };
  // Fragments of one 16-deep K half of stage ks: 4 weight and 4 token fragments per lane.
  auto read_half = [&](int ks, int kk, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
    const uint8_t* cur = lds + (ks & (kStages - 1)) * kStageBytes;
    const uint32_t coff = ((uint32_t)(2 * kk + lk) ^ lsw) << 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = *(const bf16x8*)(cur + a_row + i * 32 * kRowBytes + coff);
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = *(const bf16x8*)(cur + kOperandBytes + b_row + j * 32 * kRowBytes + coff);
  };
  auto mma_half = [&](const bf16x8 (&fa)[4], const bf16x8 (&fb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };

  // Prologue: four stages in flight, stage 0 visible, its first half read.
#pragma unroll
  for (int ks = 0; ks < kStages; ++ks)
    if (ks < nk) issue(ks);
  constexpr int per_stage = 2 * kDmaPerThread;
  if (nk >= 4)
    wait_vm_and_barrier<3 * per_stage>();
  else if (nk == 3)
    wait_vm_and_barrier<2 * per_stage>();
  else if (nk == 2)
    wait_vm_and_barrier<per_stage>();
  else
    wait_vm_and_barrier<0>();
  bf16x8 a0[4], b0[4], a1[4], b1[4];
  read_half(0, 0, a0, b0);

  // Steady state.  Each stage: the first half's 16 MFMAs issue with the second half's eight
  // fragment reads threaded between them; a barrier then makes stage ks+1 visible and frees
  // this stage's slot; the second half's MFMAs issue with the eight DMAs of stage ks+4 and the
  // next stage's first-half reads threaded between them.  Interleaving keeps the matrix pipe
  // busy while the wave issues memory instructions (one wave per SIMD has no other wave to
  // cover them), reads stay one half ahead of the MFMAs and the DMA four stages ahead.  The
  // last three stages are peeled so each wait count is a constant on a straight path.
  auto read_frag = [&](int ks, int kk, int q, bf16x8& dst) {
    const uint8_t* cur = lds + (ks & (kStages - 1)) * kStageBytes;
    const uint32_t coff = ((uint32_t)(2 * kk + lk) ^ lsw) << 4;
    dst = q < 4 ? *(const bf16x8*)(cur + a_row + q * 32 * kRowBytes + coff)
                : *(const bf16x8*)(cur + kOperandBytes + b_row + (q - 4) * 32 * kRowBytes + coff);
  };
  auto dma_one = [&](int ks, int q) {
    const uint32_t st = lds0 + (uint32_t)(ks & (kStages - 1)) * kStageBytes;
    if (q < kDmaPerThread)
      dma16(wbase + ks * kRowBytes, woff[q], st + q * 1024);
    else
      dma16(xbase + ks * kRowBytes, xoff[q - kDmaPerThread], st + kOperandBytes + (q - kDmaPerThread) * 1024);
  };
  auto mfma = [&](const bf16x8 (&fa)[4], const bf16x8 (&fb)[4], int q) {
    acc[q >> 2][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[q >> 2], fb[q & 3], acc[q >> 2][q & 3], 0, 0, 0);
  };
  auto stage = [&](int ks, auto vm_after) {
    constexpr int vm = decltype(vm_after)::value;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mfma(a0, b0, q);
      if (q < 8) read_frag(ks, 1, q, q < 4 ? a1[q] : b1[q - 4]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (vm >= 0) {
      wait_vm_and_barrier<vm>();  // stage ks+1 has landed; slot ks % 4 is free
      // A uniform test per DMA: two unrolled copies of this loop (with and without DMAs)
      // double the live ranges and spill.
      const bool more = ks + kStages < nk;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(a1, b1, q);
        if (q < 8) {
          if (more) dma_one(ks + kStages, q);
        } else {
          read_frag(ks + 1, 0, q - 8, q < 12 ? a0[q - 8] : b0[q - 12]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      mma_half(a1, b1);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  int ks = 0;
  for (; ks + 3 < nk; ++ks) stage(ks, std::integral_constant<int, 2 * per_stage>{});
  if (ks + 2 < nk) stage(ks++, std::integral_constant<int, per_stage>{});
  if (ks + 1 < nk) stage(ks++, std::integral_constant<int, 0>{});
  stage(ks, std::integral_constant<int, -1>{});
  // All waves are done reading LDS before the epilogue or the next tile reuses it.
  wait_vm_and_barrier<0>();
}

// One work item; `down` selects a down-projection tile (otherwise a fused gate/up tile).
// Each kind is its own instantiation so the register allocator sees one straight path.
// One work item.  kSplit (down tiles only) selects the K-part count at compile time: 1 = whole
// tiles, 2..4 = that many parts, 0 = any count read from the arguments.  A kernel holding
// both epilogues would keep copies of the accumulators live across the branch, and a fixed
// count lets the reduction issue the loads of several blocks of every part at once.
template <bool down, int kSplit>
__device__ __forceinline__ void producer_item(const ProducerArgs& a, uint32_t item, uint8_t* lds,
                                              uint32_t* s_last) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave: keeps bases scalar
  const int wn = wave & 1, wm = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;
  const int t = (int)((item >> kItemRowShift) & (uint32_t)(kMaxTileRows - 1));
  const int col = down ? (int)((item >> kDownColShift) & kDownColMask) : (int)(item & kItemColMask);
  const int part = down ? (int)(item & kDownPartMask) : 0;
  const TileRow tr = a.tile_rows[t];
  const int64_t H = a.H, F = a.F;
  const int e = tr.expert, lrow0 = tr.lrow0;
  // Operand rows this lane fetches: row n_i = (wave*4 + i)*16 + lane/4 of each 256-row tile.
  // Tensors stay below 4 GiB per expert/operand, so per-lane offsets fit in 32 bits and the
  // bases are wave-uniform (scalar registers).
  const uint8_t* wbase;
  const uint8_t* xbase;
  uint32_t woff[kDmaPerThread], xoff[kDmaPerThread];
  const uint32_t lrow4 = (uint32_t)lane >> 2;
  if constexpr (!down) {
    // Waves 0 and 2 fetch gate rows (W1), waves 1 and 3 the matching up rows (W3): tile rows
    // 0..63 / 128..191 are gate features, 64..127 / 192..255 the same features' up rows, so
    // each wave's MFMA quadrant holds gate and up of the same 64 features.
    wbase = (const uint8_t*)((wave & 1) ? a.w3 : a.w1) + (uint64_t)e * F * H * 2;
    xbase = (const uint8_t*)a.x;
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) {
      const uint32_t n = (uint32_t)(wave * kDmaPerThread + i) * kRowsPerDma + lrow4;
      const uint32_t ch = ((uint32_t)(lane & 3) ^ swz(n)) * 16;
      const int f = min(col * kGuTileF + (wave >> 1) * 64 + i * kRowsPerDma + (int)lrow4, (int)F - 1);
      woff[i] = (uint32_t)f * (uint32_t)H * 2 + ch;
      xoff[i] = (uint32_t)a.row_x[lrow0 + n] * (uint32_t)H * 2 + ch;
    }
  } else {
    wbase = (const uint8_t*)a.w2 + (uint64_t)e * H * F * 2;
    xbase = (const uint8_t*)a.hws + (uint64_t)lrow0 * F * 2;
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) {
      const uint32_t n = (uint32_t)(wave * kDmaPerThread + i) * kRowsPerDma + lrow4;
      const uint32_t ch = ((uint32_t)(lane & 3) ^ swz(n)) * 16;
      const int hcol = min(col * kDownTileN + (int)n, (int)H - 1);
      woff[i] = (uint32_t)hcol * (uint32_t)F * 2 + ch;
      xoff[i] = n * (uint32_t)F * 2 + ch;
    }
  }

  // K range of this item: all of it, or one of split_k near-equal runs of K steps.
  int kbeg = 0, klen = down ? (int)F : (int)H;
  constexpr bool split = kSplit != 1;
  const int S = kSplit == 0 ? a.split_k : kSplit;
  if (split) {
    const int nk = (int)F / kTileK;
    const int s0 = part * nk / S, s1 = (part + 1) * nk / S;
    kbeg = s0 * kTileK;
    klen = (s1 - s0) * kTileK;
  }
  f32x16 acc[4][4];
  tile_mma(lds, wbase + kbeg * 2, xbase + kbeg * 2, woff, xoff, klen, acc);

  if constexpr (!down) {
    // Gated activation a = bf16(silu(g) * u): lane values -> LDS tile [256 rows][128 features].
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = wm * 128 + j * 32 + lr;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int fl = wn * 64 + i * 32 + 8 * q + 4 * lk;
          const f32x16& g = acc[i][j];
          const f32x16& u = acc[i + 2][j];
          uint2 v;
          v.x = pack_bf16x2(silu_mul(g[4 * q + 0], u[4 * q + 0]), silu_mul(g[4 * q + 1], u[4 * q + 1]));
          v.y = pack_bf16x2(silu_mul(g[4 * q + 2], u[4 * q + 2]), silu_mul(g[4 * q + 3], u[4 * q + 3]));
          *(uint2*)(lds + m * kGuOutStride + fl * 2) = v;
          // Convert block by block: without this the scheduler hoists every accumulator
          // read ahead of the LDS writes and runs out of VGPRs.
          __builtin_amdgcn_sched_barrier(0);
        }
    }
    __syncthreads();
    // 16 threads store one 256-byte activation row; 16 rows per pass.
    const int c16 = tid & 15;
    const int f = col * kGuTileF + c16 * 8;
#pragma unroll 4
    for (int p = 0; p < kTileM / 16; ++p) {
      const int m = p * 16 + (tid >> 4);
      const int lrow = lrow0 + m;
      if (a.row_rank[lrow] >= 0 && f < F)  // padding rows are never read back
        *(u32x4*)(a.hws + (int64_t)lrow * F + f) = *(const u32x4*)(lds + m * kGuOutStride + c16 * 16);
    }
  } else {
    // Split K: every part stores its fp32 accumulators (in register order, so each thread
    // reads back exactly the positions it wrote) and counts itself in; the part that arrives
    // last reads all parts back and adds them in part order -- a fixed order whichever part
    // that is -- and writes the tile.  A part tile is 128 slices of 256 threads x 8 bytes:
    // slice 2b + h holds half h of accumulator block b = (i*4 + j)*4 + q.
    const int tile = t * a.down_per_row + col;
    constexpr int kPartU64 = kProducerThreads * 128;  // 8-byte elements per part tile
    const uint64_t* parts = nullptr;
    if constexpr (split) {
      parts = (const uint64_t*)a.partials + (size_t)tile * S * kPartU64;
      uint64_t* mine = (uint64_t*)a.partials + ((size_t)tile * S + part) * kPartU64 + tid;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x16& d = acc[i][j];
            const int b = (i * 4 + j) * 4 + q;
            store8_device(mine + (2 * b) * kProducerThreads, pack_f32x2(d[4 * q], d[4 * q + 1]));
            store8_device(mine + (2 * b + 1) * kProducerThreads, pack_f32x2(d[4 * q + 2], d[4 * q + 3]));
          }
      wait_vm_and_barrier<0>();  // every wave's part stores have reached the coherence point
      if (tid == 0) {
        const uint32_t prev =
            __hip_atomic_fetch_add(&a.arrivals[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *s_last = (prev + 1 == (uint32_t)S) ? 1u : 0u;
      }
      __syncthreads();
      if (*s_last == 0) return;  // another part finishes the tile
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    // Down-projection output: lane values -> LDS tile [256 rows][256 hidden columns].
    auto stage_out = [&](int i, int j, int q, float4 s) {
      const int m = wm * 128 + j * 32 + lr;
      const int nl = wn * 128 + i * 32 + 8 * q + 4 * lk;
      uint2 v;
      v.x = pack_bf16x2(s.x, s.y);
      v.y = pack_bf16x2(s.z, s.w);
      *(uint2*)(lds + m * kDownOutStride + nl * 2) = v;
    };
    // Accumulator block b of part p: its two 8-byte halves, widened back to four floats.
    auto part_block = [&](const uint64_t* src, int p, int b) {
      const uint64_t lo = src[(size_t)p * kPartU64 + (2 * b) * kProducerThreads];
      const uint64_t hi = src[(size_t)p * kPartU64 + (2 * b + 1) * kProducerThreads];
      return float4{__uint_as_float((uint32_t)lo), __uint_as_float((uint32_t)(lo >> 32)),
                    __uint_as_float((uint32_t)hi), __uint_as_float((uint32_t)(hi >> 32))};
    };
    if constexpr (kSplit == 0) {
      // Any part count: blocks b = (i*4 + j)*4 + q indexed at run time, every part read back.
      const uint64_t* src = parts + tid;
#pragma unroll 1
      for (int b = 0; b < 64; ++b) {
        float4 s = part_block(src, 0, b);
        for (int p = 1; p < S; ++p) {
          const float4 v = part_block(src, p, b);
          s.x += v.x;
          s.y += v.y;
          s.z += v.z;
          s.w += v.w;
        }
        stage_out(b >> 4, (b >> 2) & 3, b & 3, s);
      }
    } else if constexpr (split) {
      // kSplit parts: all parts read back (this part's too: the same values, and no branch
      // that would serialize the loads), 4 blocks of kSplit parts in flight per step.
      const uint64_t* src = parts + tid;
      constexpr int kGroup = kSplit == 3 ? 2 : 4;  // keeps 4*kGroup*kSplit loaded floats live
#pragma unroll 1
      for (int b0 = 0; b0 < 64; b0 += kGroup) {
        float4 v[kGroup][kSplit];
#pragma unroll
        for (int u = 0; u < kGroup; ++u)
#pragma unroll
          for (int p = 0; p < kSplit; ++p) v[u][p] = part_block(src, p, b0 + u);
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          float4 s = v[u][0];
#pragma unroll
          for (int p = 1; p < kSplit; ++p) {
            s.x += v[u][p].x;
            s.y += v[u][p].y;
            s.z += v[u][p].z;
            s.w += v[u][p].w;
          }
          const int b = b0 + u;
          stage_out(b >> 4, (b >> 2) & 3, b & 3, s);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x16& d = acc[i][j];
            stage_out(i, j, q, float4{d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]});
            __builtin_amdgcn_sched_barrier(0);  // block by block (see above)
          }
    }
    __syncthreads();
    // Rows returning to another rank go to the staged output Y (the consumer moves them);
    // local rows go straight to the local receive buffer when the producer writes them
    // directly.  In a signalled launch a wave stores one 512-byte row (64 lanes x 8 bytes, 4
    // rows per pass) and the Y rows at device scope, so publishing the tile needs no L2
    // writeback.  Without signalling, 32 lanes store a row with ordinary 16-byte stores; in
    // the no-consumer ablation every row goes straight to its receive buffer.
    const bool direct = (a.mode & kModeLocalDirect) != 0;
    const bool signal = (a.mode & kModeSignal) != 0;
    if (signal) {
      const int c8 = tid & 63;
      const int n = col * kDownTileN + c8 * 4;
#pragma unroll 4
      for (int p = 0; p < kTileM / 4; ++p) {
        const int m = p * 4 + (tid >> 6);
        const int lrow = lrow0 + m;
        const int rank = a.row_rank[lrow];
        if (rank >= 0 && n < H) {
          const uint64_t v = *(const uint64_t*)(lds + m * kDownOutStride + c8 * 8);
          if (direct && rank == a.self_rank)
            *(__attribute__((address_space(1))) uint64_t*)(a.ret[rank] + (int64_t)a.row_slot[lrow] * H + n) = v;
          else
            store8_device(a.y + (int64_t)lrow * H + n, v);
        }
      }
    } else {
      const bool direct_all = (a.mode & kModeDirectAll) != 0;
      const int c16 = tid & 31;
      const int n = col * kDownTileN + c16 * 8;
#pragma unroll 4
      for (int p = 0; p < kTileM / 8; ++p) {
        const int m = p * 8 + (tid >> 5);
        const int lrow = lrow0 + m;
        const int rank = a.row_rank[lrow];
        if (rank >= 0 && n < H) {
          const u32x4 v = *(const u32x4*)(lds + m * kDownOutStride + c16 * 16);
          if (direct_all || (direct && rank == a.self_rank))
            *(g_u32x4*)(a.ret[rank] + (int64_t)a.row_slot[lrow] * H + n) = v;
          else
            *(g_u32x4*)(a.y + (int64_t)lrow * H + n) = v;
        }
      }
    }
    // Every wave's output stores have completed (the staged rows at the coherence point)
    // before wave 0 raises the flag; a plain barrier does not wait for other waves' stores.
    wait_vm_and_barrier<0>();
    if (signal && (tr.has_remote || !direct)) {
      if (tid == 0) __hip_atomic_store(&a.flags[tile], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Persistent producer: every workgroup claims items from this launch's queue until it is
// empty.  Nothing inside waits on another workgroup, so progress never depends on which
// workgroups are resident.
template <bool down, int kSplit>
__global__ __launch_bounds__(kProducerThreads, 1) void producer_kernel(ProducerArgs a) {
  static_assert(kLdsAlloc >= kLdsBytes, "staging must fit the LDS allocation");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsAlloc];
  __shared__ uint32_t s_next, s_last;
  const int tid = threadIdx.x;
  if (tid == 0) {
    s_next = atomicAdd(a.claim, 1u);
    if (s_next < (uint32_t)a.n_items) atomicAdd(a.active, 1u);
  }
  __syncthreads();
  uint32_t cur = __builtin_amdgcn_readfirstlane(s_next);  // uniform: item fields stay scalar
  while (cur < (uint32_t)a.n_items) {
    __syncthreads();
    // Claim the next item now; its index is read after this one finishes.
    if (tid == 0) s_next = atomicAdd(a.claim, 1u);
    producer_item<down, kSplit>(a, a.items[cur], lds, &s_last);
    __syncthreads();
    cur = __builtin_amdgcn_readfirstlane(s_next);
  }
}

// ---------------------------------------------------------------------------
// Consumer: claim segments in ready order; wave 0 polls the segment's flags
// (one flag per lane, all lanes must read the current epoch), then the whole
// workgroup copies rows * H bf16 with 16-byte loads and stores.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kConsumerThreads, kConsumerMinWaves) void consumer_kernel(ConsumerArgs a) {
  __shared__ int32_t s_seg;
  __shared__ uint32_t s_abort;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t polls = 0, waited = 0;
  for (;;) {
    if (tid == 0) {
      s_seg = (int32_t)atomicAdd(&a.ctr->seg_next, 1u);
      s_abort = 0;
    }
    __syncthreads();
    const int32_t s = s_seg;
    if (s >= a.n_segs) break;
    const Segment sg = a.segs[s];
    if (wave == 0) {
      const uint64_t t0 = ticks();
      bool expired = false;
      for (int base = 0; base < sg.flag_count && !expired; base += 64) {
        const bool mine = base + lane < sg.flag_count;
        const uint32_t* fp = a.flags + sg.flag_begin + base + lane;
        for (;;) {
          const uint32_t v =
              mine ? __hip_atomic_load(fp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : a.epoch;
          if (__all(v == a.epoch)) break;
          ++polls;
          if (ticks() - t0 > a.watchdog_ticks) {
            expired = true;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      waited += ticks() - t0;
      if (expired && lane == 0) s_abort = 1;
    }
    __syncthreads();
    if (s_abort) {
      if (tid == 0) {
        __hip_atomic_fetch_add(&a.ctr->timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_or(&a.ctr->timeout_where, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      break;
    }
    // The segment is contiguous on both sides: a flat 16-byte-vector copy in chunks of
    // kCopyUnroll vectors per thread, double-buffered: the next chunk's loads are in flight
    // while the current chunk is stored, so neither load nor store latency is exposed per
    // chunk.  The last chunk re-reads itself as its "next" (in bounds) instead of branching,
    // which would drain every outstanding access.
    const u32x4* src = (const u32x4*)(a.y + (int64_t)sg.y_row0 * a.H);
    g_u32x4* dst = (g_u32x4*)(a.ret[sg.dst_rank] + (int64_t)sg.slot0 * a.H);
    const int64_t n16 = (int64_t)sg.rows * a.H / 8;
    constexpr int kU = kCopyUnroll;
    constexpr int64_t kStep = (int64_t)kU * kConsumerThreads;
    const int64_t nfull = n16 / kStep;
    if (nfull > 0) {
      u32x4 cur[kU], nxt[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) cur[u] = src[tid + u * kConsumerThreads];
      for (int64_t c = 0; c < nfull; ++c) {
        const int64_t base = c * kStep + tid;
        const int64_t next = (c + 1 < nfull ? c + 1 : c) * kStep + tid;
#pragma unroll
        for (int u = 0; u < kU; ++u) nxt[u] = src[next + u * kConsumerThreads];
#pragma unroll
        for (int u = 0; u < kU; ++u) dst[base + u * kConsumerThreads] = cur[u];
#pragma unroll
        for (int u = 0; u < kU; ++u) cur[u] = nxt[u];
      }
    }
    for (int64_t i = nfull * kStep + tid; i < n16; i += kConsumerThreads) dst[i] = src[i];
    __syncthreads();
  }
  if (wave == 0 && lane == 0 && (polls || waited)) {
    atomicAdd((unsigned long long*)&a.ctr->poll_iters, (unsigned long long)polls);
    atomicAdd((unsigned long long*)&a.ctr->wait_ticks, (unsigned long long)waited);
  }
}

// ---------------------------------------------------------------------------
// Baseline bulk return: every routed row of the staged output to its slot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a) {
  const int64_t per_row = a.H / 8;
  for (int64_t r = blockIdx.x; r < a.n_lrows; r += gridDim.x) {
    const int rank = a.row_rank[r];
    if (rank < 0) continue;
    const u32x4* src = (const u32x4*)(a.y + r * a.H);
    g_u32x4* dst = (g_u32x4*)(a.ret[rank] + (int64_t)a.row_slot[r] * a.H);
    for (int64_t i = threadIdx.x; i < per_row; i += blockDim.x) dst[i] = src[i];
  }
}

__global__ __launch_bounds__(256) void init_kernel(InitArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i == 0) {
    a.ctr->gu_next = 0;
    a.ctr->down_next = 0;
    a.ctr->seg_next = 0;
    a.ctr->gu_active = 0;
    a.ctr->down_active = 0;
    a.ctr->poll_iters = 0;
    a.ctr->wait_ticks = 0;
  }
  for (int64_t j = i; j < a.n_arrivals; j += stride) a.arrivals[j] = 0;
  if (a.poison) {
    const u32x4 nan = {0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};
    for (int64_t j = i; j < a.poison_elems / 8; j += stride) ((u32x4*)a.poison)[j] = nan;
  }
}

hipError_t launch_init(const InitArgs& a, hipStream_t s) {
  int grid = 64;
  if (a.poison) grid = 1024;
  hipLaunchKernelGGL(init_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_producer(const ProducerArgs& a, bool down, int grid, hipStream_t s) {
  const dim3 g(grid), b(kProducerThreads);
  if (!down)
    hipLaunchKernelGGL((producer_kernel<false, 1>), g, b, 0, s, a);
  else if (a.split_k == 1)
    hipLaunchKernelGGL((producer_kernel<true, 1>), g, b, 0, s, a);
  else if (a.split_k == 2)
    hipLaunchKernelGGL((producer_kernel<true, 2>), g, b, 0, s, a);
  else if (a.split_k == 3)
    hipLaunchKernelGGL((producer_kernel<true, 3>), g, b, 0, s, a);
  else if (a.split_k == 4)
    hipLaunchKernelGGL((producer_kernel<true, 4>), g, b, 0, s, a);
  else
    hipLaunchKernelGGL((producer_kernel<true, 0>), g, b, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_consumer(const ConsumerArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(consumer_kernel, dim3(grid), dim3(kConsumerThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_scatter(const ScatterArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(scatter_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

int producer_blocks_per_cu() {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, producer_kernel<false, 1>, kProducerThreads, 0) != hipSuccess)
    return 1;
  return n > 0 ? n : 1;
}

}  // namespace moe
