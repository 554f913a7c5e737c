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
#include <limits.h>
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
// Word 3 of a raw buffer resource on gfx9-family GPUs (stride 0, byte-addressed, range-checked).
constexpr int kBufferRsrcWord3 = 0x00020000;

// Operand blocks in LDS: 256 rows x 64 k (bf16) = 32 KiB, 128 bytes per row -- one whole
// cache line of the row-major operand, so every line a K step touches is used in full (with
// 64-byte rows each line is fetched twice, and the load path then streams about 0.6x as many
// useful bytes per clock).  A K step needs a weight block and a token block; a ring of five
// blocks (all 160 KiB of LDS) keeps one and a half K steps of loads in flight.  Global
// memory is copied straight into LDS with global_load_lds_dwordx4 (no register staging).
// A DMA instruction writes 64 lanes x 16 bytes contiguously, i.e. 8 rows, so each lane
// fetches the 16-byte chunk that belongs at its slot: chunk c of row r sits at physical
// chunk c ^ swz(r).
constexpr int kRowBytes = kTileK * 2;                  // 128
constexpr int kBlockBytes = kTileM * kRowBytes;        // 32 KiB: one operand of one K step
constexpr int kRingBlocks = 5;
constexpr int kLdsBytes = kRingBlocks * kBlockBytes;   // 160 KiB: the whole LDS of a CU
constexpr int kRowsPerDma = 64 * 16 / kRowBytes;       // 8 rows per DMA instruction
constexpr int kDmaPerThread = kTileM / kRowsPerDma / 4;  // 8 per operand block per thread
// Epilogue staging: the finished tile goes through LDS (free once the pipeline drains) so
// that global stores are whole 16-byte chunks of contiguous rows.  Rows are padded by 16
// bytes so the 32 lanes writing one column of 32 rows hit distinct banks.
constexpr int kDownOutStride = kDownTileN * 2 + 16;    // 528 B per staged output row
constexpr int kGuOutStride = kGuTileF * 2 + 16;        // 272 B per staged activation row
// Words past both staging areas carry the next work item (its queue position, item word and
// tile row) and the split-K verdict between the waves; the operand ring overwrites them, so
// they are used only while the ring is idle (the epilogue and the item boundary).
constexpr int kSharedWords = kLdsBytes - 48;
constexpr int kWordPos = 0, kWordSplit = 1, kWordItem = 2, kWordTileRow = 3;  // tile row: 6 words
static_assert((kWordTileRow + 6) * 4 <= kLdsBytes - kSharedWords, "shared words");
static_assert(kTileM * kDownOutStride <= kSharedWords, "down staging overlaps the shared words");
// Down epilogue: each tile row's (rank, slot) pairs, right past the staged output tile.
constexpr int kDownRowInfo = kTileM * kDownOutStride;
static_assert(kDownRowInfo + kTileM * 8 <= kSharedWords, "row info overlaps the shared words");
static_assert(kTileM * kGuOutStride <= kSharedWords, "gate/up staging overlaps the shared words");

// Chunk swizzle of the 128-byte operand rows: chunk c of row r is stored at c ^ ((r / 2) % 8).
// A fragment read (ds_read_b128) is served 16 lanes at a time; those lanes read one chunk
// column of 16 consecutive rows, and with 64 four-byte banks (256 bytes) even and odd rows
// fall in opposite bank halves, so the XOR spreads the 16 reads over all 16 bank groups.
__device__ __forceinline__ uint32_t swz(uint32_t row) { return (row >> 1) & 7u; }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// silu(g) * u = g * u / (1 + e^-g), with the hardware exponential and reciprocal: each is within
// about one fp32 ulp, far below the bf16 rounding that follows, where an IEEE division costs ten
// instructions per element in an epilogue that otherwise leaves the matrix cores idle.  Large
// negative g gives e^-g = inf, a reciprocal of 0 and a result of 0, as the exact formula does.
__device__ __forceinline__ float silu_mul(float g, float u) {
  return (g * u) * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

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

// MOE_WRITE_COUNTS: counts `words` 8-byte words stored into the receive buffer for logical row lrow.
__device__ __forceinline__ void count_words(uint32_t* wcount, int64_t lrow, uint32_t words) {
  if (wcount) __hip_atomic_fetch_add(&wcount[lrow], words, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

// Rows of one operand as a DMA source.  Instruction i of a wave fetches the 8 rows starting at
// g_i = min(g0 + 8i, gmax) from the wave-uniform address base + g_i * stride; each lane adds
// lane_off[i % 2]: its row (lane / 8) times the stride plus its swizzled 16-byte chunk (the
// swizzle of rows wave*64 + i*8 + lane/8 depends on i only through i % 2).  H and F are
// multiples of 64, so an 8-row group lies wholly inside or wholly past the operand's last
// row, and clamping the group start keeps every read in bounds.
struct DmaRows {
  const uint8_t* base;
  uint32_t stride;
  int32_t g0, gmax;
  uint32_t lane_off[2];
  uint32_t step;  // bytes from one K step of a row to the next (128 when rows are K-contiguous)
  __device__ __forceinline__ const uint8_t* rows(int i) const {
    return base + (uint64_t)(uint32_t)min(g0 + 8 * i, gmax) * stride;
  }
};

// Lane offset of row lane/8 with its swizzled chunk, for even (p = 0) or odd (p = 1) DMA
// instructions: the tile row is wave*64 + i*8 + lane/8, whose swizzle is (4*(i%2) + lane/16) % 8.
__device__ __forceinline__ uint32_t dma_lane_off(int lane, int p, uint32_t stride) {
  const uint32_t r = (uint32_t)lane >> 3;
  return r * stride + (((uint32_t)(lane & 7) ^ ((4u * p + (r >> 1)) & 7u)) << 4);
}

// ---------------------------------------------------------------------------
// One 256x256 output tile: acc[i][j] holds D[n][m] for the wave's 128x128
// quadrant, n = wn*128 + i*32 + 8*(r/4) + 4*(lane/32) + r%4, m = wm*128 + j*32 + lane%32.
// DMA instruction i of a wave fills operand-tile rows wave*64 + i*8 .. +7 (w for the weight
// tile, x for the token tile); with kGatherX the token rows are gathered, xoff[i] being this
// lane's byte offset from x.base for instruction i.
//
// Block b of the ring holds the weights (b even) or tokens (b odd) of K step b/2, in slot
// b % 5.  Prologue: blocks 0-3 in flight.  K step ks runs four 16-deep MFMA sub-steps; each
// sub-step's 16 MFMAs issue with the next sub-step's 8 fragment reads threaded between them,
// and with the DMAs of the blocks whose slots are free: block 2ks+4 during sub-step 0 (its
// slot held K step ks-1's tokens), block 2ks+5 during sub-step 3, after the barrier that
// ends every wave's reads of step ks.  That barrier also waits for step ks+1's blocks, with
// only block 2ks+4 allowed in flight.  The last two K steps are peeled so each wait count
// is a constant on a straight path.
// ---------------------------------------------------------------------------
template <bool kGatherX, class Late>
__device__ __forceinline__ void tile_mma(uint8_t* __restrict__ lds, const DmaRows& w, const DmaRows& x,
                                         const uint32_t (&xoff)[kDmaPerThread], int K, f32x16 (&acc)[4][4],
                                         Late&& late) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave & 1, wm = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;
  const uint32_t lsw = swz(lr);  // rows wn*128 + i*32 + lr share lr's swizzle
  const uint32_t a_row = (uint32_t)(wn * 128 + lr) * kRowBytes;
  const uint32_t b_row = (uint32_t)(wm * 128 + lr) * kRowBytes;
  const uint32_t dma_off = (uint32_t)wave * kDmaPerThread * 1024;

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  const int nk = K / kTileK;
  const uint32_t lds0 = lds_addr(lds) + dma_off;
  auto slot = [](int blk) { return (uint32_t)(blk % kRingBlocks) * kBlockBytes; };
  auto dma_w = [&](int ks, int q) {
    dma16(w.rows(q) + (size_t)ks * w.step, w.lane_off[q & 1], lds0 + slot(2 * ks) + q * 1024);
  };
  auto dma_x = [&](int ks, int q) {
    if constexpr (kGatherX)
      dma16(x.base + (size_t)ks * x.step, xoff[q], lds0 + slot(2 * ks + 1) + q * 1024);
    else
      dma16(x.rows(q) + (size_t)ks * x.step, x.lane_off[q & 1], lds0 + slot(2 * ks + 1) + q * 1024);
  };
  // Fragment q of sub-step kk of K step ks: q < 4 weight rows, else token rows.  The lane
  // reads logical chunk 2kk + lk of its row, stored at chunk (2kk + lk) ^ lsw = (lk ^ lsw) ^ 2kk;
  // slot and row offsets are multiples of 128, so the sub-step enters as an XOR of bits 5-6
  // of one per-operand base and the 32-row block as an immediate offset.
  const uint32_t a_lane = a_row + (((uint32_t)lk ^ lsw) << 4);
  const uint32_t b_lane = b_row + (((uint32_t)lk ^ lsw) << 4);
  auto read_frag = [&](int ks, int kk, int q, bf16x8& dst) {
    const uint32_t base = q < 4 ? a_lane + slot(2 * ks) : b_lane + slot(2 * ks + 1);
    dst = *(const bf16x8*)(lds + ((base ^ ((uint32_t)kk << 5)) + (q & 3) * 32 * kRowBytes));
  };
  auto mfma = [&](const bf16x8 (&fa)[4], const bf16x8 (&fb)[4], int q) {
    acc[q >> 2][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[q >> 2], fb[q & 3], acc[q >> 2][q & 3], 0, 0, 0);
  };

  // Prologue: K steps 0 and 1 in flight, step 0 visible, its first sub-step read.
#pragma unroll
  for (int q = 0; q < kDmaPerThread; ++q) dma_w(0, q);
#pragma unroll
  for (int q = 0; q < kDmaPerThread; ++q) dma_x(0, q);
  if (nk > 1) {
#pragma unroll
    for (int q = 0; q < kDmaPerThread; ++q) dma_w(1, q);
#pragma unroll
    for (int q = 0; q < kDmaPerThread; ++q) dma_x(1, q);
    wait_vm_and_barrier<2 * kDmaPerThread>();
  } else {
    wait_vm_and_barrier<0>();
  }
  bf16x8 a0[4], b0[4], a1[4], b1[4];
#pragma unroll
  for (int q = 0; q < 8; ++q) read_frag(0, 0, q, q < 4 ? a0[q] : b0[q - 4]);

  // kind 0: steady step (DMAs, then wait with one block in flight); 1: next to last (no
  // DMAs, wait for everything); 2: last step (no wait, nothing to read ahead).
  auto step = [&](int ks, auto kind) {
    constexpr int kd = decltype(kind)::value;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mfma(a0, b0, q);
      if (q & 1)
        read_frag(ks, 1, q >> 1, (q >> 1) < 4 ? a1[q >> 1] : b1[(q >> 1) - 4]);
      else if constexpr (kd == 0)
        dma_w(ks + 2, q >> 1);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mfma(a1, b1, q);
      if (q < 8) read_frag(ks, 2, q, q < 4 ? a0[q] : b0[q - 4]);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mfma(a0, b0, q);
      if (q < 8) read_frag(ks, 3, q, q < 4 ? a1[q] : b1[q - 4]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (kd < 2) {
      wait_vm_and_barrier<kd == 0 ? kDmaPerThread : 0>();  // step ks+1 visible, step ks's slots free
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(a1, b1, q);
        if (q & 1)
          read_frag(ks + 1, 0, q >> 1, (q >> 1) < 4 ? a0[q >> 1] : b0[(q >> 1) - 4]);
        else if constexpr (kd == 0)
          dma_x(ks + 2, q >> 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        mfma(a1, b1, q);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  int ks = 0;
  for (; ks + 2 < nk; ++ks) step(ks, std::integral_constant<int, 0>{});
  late();  // two K steps (or one) before the end
  if (ks + 1 < nk) step(ks++, std::integral_constant<int, 1>{});
  step(ks, std::integral_constant<int, 2>{});
  // All waves are done reading LDS before the epilogue or the next tile reuses it.
  wait_vm_and_barrier<0>();
}

// One work item; `down` selects a down-projection tile (otherwise a fused gate/up tile).
// Each kind is its own instantiation so the register allocator sees one straight path.
// One work item.  kSplit (down tiles only) selects the K-part count at compile time: 1 = whole
// tiles, 2..4 = that many parts, 0 = the count of the item's tile row.  A kernel holding
// both epilogues would keep copies of the accumulators live across the branch, and a fixed
// count lets the reduction issue the loads of several blocks of every part at once.
//
// `hook()` runs once the epilogue has staged the tile (not on the paths that return early):
// thread 0 fetches the next item's descriptor there, and the stores that follow hide part of
// the load latency.  (Branching there while the accumulators are still live, right after the
// K loop, made the compiler spill them.)
template <bool down, int kSplit, class Late, class Hook>
__device__ __forceinline__ void producer_item(const ProducerArgs& a, uint32_t item, const TileRow& tr,
                                              uint8_t* lds, uint32_t* words, Late&& late, Hook&& hook) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave: keeps bases scalar
  const int wn = wave & 1, wm = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;
  const int t = (int)((item >> kItemRowShift) & (uint32_t)(kMaxTileRows - 1));
  const int col = down ? (int)((item >> kDownColShift) & kDownColMask) : (int)(item & kItemColMask);
  const int part = down ? (int)(item & kDownPartMask) : 0;
  const int64_t H = a.H, F = a.F;
  const int e = tr.expert, lrow0 = tr.lrow0;
  // Operand rows: DMA instruction i of a wave fills tile rows wave*64 + i*8 .. +7.  Tensors
  // stay below 4 GiB per expert/operand, so per-lane offsets fit in 32 bits and the bases are
  // wave-uniform (scalar registers).
  DmaRows w, x;
  uint32_t xoff[kDmaPerThread];
  if constexpr (!down) {
    // Waves 0 and 2 fetch gate rows (W1), waves 1 and 3 the matching up rows (W3): tile rows
    // 0..63 / 128..191 are gate features, 64..127 / 192..255 the same features' up rows, so
    // each wave's MFMA quadrant holds gate and up of the same 64 features.
    const uint32_t stride = (uint32_t)H * 2;
    w.base = (const uint8_t*)((wave & 1) ? a.w3 : a.w1) + (uint64_t)e * F * H * 2;
    w.stride = stride;
    w.g0 = col * kGuTileF + (wave >> 1) * 64;
    w.gmax = (int)F - kRowsPerDma;
    w.lane_off[0] = dma_lane_off(lane, 0, stride);
    w.lane_off[1] = dma_lane_off(lane, 1, stride);
    w.step = kRowBytes;
    // Token rows are gathered from the dispatched rows through row_x.
    x.base = (const uint8_t*)a.x;
    x.step = kRowBytes;
    const uint32_t r = (uint32_t)lane >> 3;
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) {
      const uint32_t n = (uint32_t)(wave * kDmaPerThread + i) * kRowsPerDma + r;
      // 24-bit multiply (rows < 2^24, stride <= 2^17): a 32-bit result, where a full multiply-add
      // would produce register pairs whose high halves stay allocated.
      xoff[i] = __umul24((uint32_t)a.row_x[lrow0 + n], stride) + (((uint32_t)(lane & 7) ^ swz(n)) << 4);
    }
    // The offsets are complete before the first operand DMA.  The compiler counts only its own
    // loads, not the DMAs: had it waited for each offset just before its token DMA, each of
    // those waits would also have drained the weight DMAs issued in between, serialising the
    // prologue into three memory latencies instead of two.
#pragma unroll
    for (int i = 0; i < kDmaPerThread; ++i) asm volatile("" ::"v"(xoff[i]));
  } else {
    const uint32_t stride = (uint32_t)F * 2;
    w.base = (const uint8_t*)a.w2 + (uint64_t)e * H * F * 2;
    w.stride = stride;
    w.g0 = col * kDownTileN + wave * 64;
    w.gmax = (int)H - kRowsPerDma;
    w.lane_off[0] = dma_lane_off(lane, 0, stride);
    w.lane_off[1] = dma_lane_off(lane, 1, stride);
    w.step = kRowBytes;
    // Token rows are the tile row's own activation rows in the K-blocked workspace: the 256
    // rows' 64 features of one K step are one contiguous 32 KiB block.
    x.base = (const uint8_t*)a.hws + (uint64_t)lrow0 * kRowBytes;
    x.stride = kRowBytes;
    x.g0 = wave * 64;
    x.gmax = kTileM - kRowsPerDma;
    x.lane_off[0] = dma_lane_off(lane, 0, kRowBytes);
    x.lane_off[1] = dma_lane_off(lane, 1, kRowBytes);
    x.step = (uint32_t)a.hws_rows * kRowBytes;
  }

  // K range of this item: all of it, or one of split_k near-equal runs of K steps.
  int kbeg = 0, klen = down ? (int)F : (int)H;
  constexpr bool split = kSplit != 1;
  const int S = kSplit == 0 ? tr.split : kSplit;
  if (split) {
    const int nk = (int)F / kTileK;
    const int s0 = part * nk / S, s1 = (part + 1) * nk / S;
    kbeg = s0 * kTileK;
    klen = (s1 - s0) * kTileK;
  }
  f32x16 acc[4][4];
  w.base += (size_t)(kbeg / kTileK) * w.step;
  x.base += (size_t)(kbeg / kTileK) * x.step;
  tile_mma<!down>(lds, w, x, xoff, klen, acc, late);

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
    hook();
    // 16 threads store one row's 128 features: 8 threads per 64-feature K block of the
    // workspace [F / 64][hws_rows][64], so consecutive rows fill contiguous 128-byte runs.
    const int c16 = tid & 15;
    const int f = col * kGuTileF + c16 * 8;
    uint16_t* blk = a.hws + ((size_t)(f / kTileK) * a.hws_rows) * kTileK + (f % kTileK);
    // Padding rows are stored too: they gather a valid token row, so their activations are
    // finite, and the down launch only uses them for padding outputs it never stores -- no
    // per-row lookup sits between the staged tile and its stores.
    if (f < F) {
#pragma unroll 4
      for (int p = 0; p < kTileM / 16; ++p) {
        const int m = p * 16 + (tid >> 4);
        *(u32x4*)(blk + (size_t)(lrow0 + m) * kTileK) = *(const u32x4*)(lds + m * kGuOutStride + c16 * 16);
      }
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
      const size_t first = (size_t)tr.part_base + (size_t)col * S;  // this tile's part 0
      parts = (const uint64_t*)a.partials + first * kPartU64;
      uint64_t* mine = (uint64_t*)a.partials + (first + part) * kPartU64 + tid;
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
      if (kSplit == 0 && (a.mode & kModeDeferTail)) return;  // the tail kernel adds the parts
      wait_vm_and_barrier<0>();  // every wave's part stores have reached the coherence point
      if (tid == 0) {
        const uint32_t prev =
            __hip_atomic_fetch_add(&a.arrivals[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        words[kWordSplit] = (prev + 1 == (uint32_t)S) ? 1u : 0u;
      }
      __syncthreads();
      if (words[kWordSplit] == 0) return;  // another part finishes the tile
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    // Each row's rank and slot for the stores below: one row per thread, loaded now so the
    // loads overlap the staging, and put in LDS past the staged tile.
    static_assert(kProducerThreads == kTileM, "one row per thread");
    const int my_rank = a.row_rank[lrow0 + tid], my_slot = a.row_slot[lrow0 + tid];
    int32_t* rinfo = (int32_t*)(lds + kDownRowInfo);
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
      // Any part count: 2 blocks at a time, their parts read back 4 at a time with every
      // load of a round issued together (a part past the count re-reads the last part and
      // is not added), and added in part order.
      const uint64_t* src = parts + tid;
      constexpr int kB = 2, kP = 4;
#pragma unroll 1
      for (int b0 = 0; b0 < 64; b0 += kB) {
        float4 acc4[kB];
#pragma unroll 1
        for (int p0 = 0; p0 < S; p0 += kP) {
          float4 v[kB][kP];
#pragma unroll
          for (int u = 0; u < kB; ++u)
#pragma unroll
            for (int pp = 0; pp < kP; ++pp) v[u][pp] = part_block(src, min(p0 + pp, S - 1), b0 + u);
#pragma unroll
          for (int u = 0; u < kB; ++u)
#pragma unroll
            for (int pp = 0; pp < kP; ++pp) {
              const int p = p0 + pp;
              if (p == 0) {
                acc4[u] = v[u][pp];
              } else if (p < S) {
                acc4[u].x += v[u][pp].x;
                acc4[u].y += v[u][pp].y;
                acc4[u].z += v[u][pp].z;
                acc4[u].w += v[u][pp].w;
              }
            }
        }
#pragma unroll
        for (int u = 0; u < kB; ++u) {
          const int b = b0 + u;
          stage_out(b >> 4, (b >> 2) & 3, b & 3, acc4[u]);
        }
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
    rinfo[2 * tid] = my_rank;
    rinfo[2 * tid + 1] = my_slot;
    __syncthreads();
    hook();
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
        const int rank = rinfo[2 * m];
        if (rank >= 0 && n < H) {
          const uint64_t v = *(const uint64_t*)(lds + m * kDownOutStride + c8 * 8);
          if (direct && rank == a.self_rank) {
            *(__attribute__((address_space(1))) uint64_t*)(a.ret[rank] + (int64_t)rinfo[2 * m + 1] * H + n) = v;
            count_words(a.wcount, lrow, 1);
          } else {
            store8_device(a.y + (int64_t)lrow * H + n, v);
          }
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
        const int rank = rinfo[2 * m];
        if (rank >= 0 && n < H) {
          const u32x4 v = *(const u32x4*)(lds + m * kDownOutStride + c16 * 16);
          if (direct_all || (direct && rank == a.self_rank)) {
            *(g_u32x4*)(a.ret[rank] + (int64_t)rinfo[2 * m + 1] * H + n) = v;
            count_words(a.wcount, lrow, 2);
          } else {
            *(g_u32x4*)(a.y + (int64_t)lrow * H + n) = v;
          }
        }
      }
    }
    // Every wave's output stores have completed (the staged rows at the coherence point)
    // before wave 0 raises the flag; a plain barrier does not wait for other waves' stores.
    // A tile that raises no flag does not wait: its stores drain under the next item's first
    // operand loads (the staged tile in LDS is free once the loop's barrier has passed, every
    // wave's LDS reads for its stores having returned).
    if (signal && (tr.has_remote || !direct)) {
      wait_vm_and_barrier<0>();
      if (tid == 0) {
        if (a.tile_ready) a.tile_ready[tile] = ticks();
        __hip_atomic_store(&a.flags[tile], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// The XCD (accelerator die) this wave runs on: hardware register XCC_ID, bits 3:0.
__device__ __forceinline__ uint32_t xcc_id() {
  constexpr int kHwRegXccId = 20;
  return (uint32_t)__builtin_amdgcn_s_getreg(kHwRegXccId | (0 << 6) | ((4 - 1) << 11)) & (kXcds - 1);
}

// The wave's HW_ID register: wave slot, SIMD, compute unit, shader array and shader engine.
__device__ __forceinline__ uint32_t hw_id() {
  constexpr int kHwRegHwId = 4;
  return (uint32_t)__builtin_amdgcn_s_getreg(kHwRegHwId | (0 << 6) | ((32 - 1) << 11));
}

// A load through the scalar cache: the plan arrays are written before the launch and only read
// during it.  Scalar loads count on lgkmcnt, so waiting for one does not also wait for the vector
// stores issued before it (vmcnt counts loads and stores in issue order).
template <class T>
__device__ __forceinline__ T load_scalar(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}

// Claims the next item of this launch (thread 0): from queue q first when try_q (the workgroup's
// own XCD's queue, or the one it last took from), else from the first queue at or after q that
// still holds items.  Returns the item's position in a.items, or `end` once every queue is empty.
// The queues' claim counts are read together, one round trip, instead of one atomic per empty
// queue in turn: at a launch's end every workgroup learns that all queues are empty in one round
// trip, not eight.  Counts only grow, so a queue seen exhausted stays exhausted; each failed claim
// exhausts one more queue, so the loop ends within kXcds + 1 passes.
__device__ __forceinline__ uint32_t claim_item(const ProducerArgs& a, uint32_t& q, uint32_t end, bool try_q) {
  if (try_q) {
    const uint32_t i = atomicAdd(&a.claim[q], 1u);
    const int32_t q0 = a.queue[q], q1 = a.queue[q + 1];
    if (i < (uint32_t)(q1 - q0)) return (uint32_t)q0 + i;
  }
  int32_t bound[kXcds + 1];
#pragma unroll
  for (int x = 0; x <= kXcds; ++x) bound[x] = load_scalar(a.queue + x);
  for (int pass = 0; pass <= kXcds; ++pass) {
    uint32_t cnt[kXcds];
#pragma unroll
    for (int x = 0; x < kXcds; ++x) cnt[x] = __hip_atomic_load(&a.claim[x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t open = 0;
#pragma unroll
    for (int x = 0; x < kXcds; ++x) open |= (cnt[x] < (uint32_t)(bound[x + 1] - bound[x]) ? 1u : 0u) << x;
    if (open == 0) return end;
    const uint32_t rot = ((open >> q) | (open << (kXcds - q))) & ((1u << kXcds) - 1);
    const uint32_t x = (q + (uint32_t)__builtin_ctz(rot)) & (kXcds - 1);
    int32_t x0 = bound[0], x1 = bound[1];
#pragma unroll
    for (int y = 1; y < kXcds; ++y)
      if ((uint32_t)y == x) {
        x0 = bound[y];
        x1 = bound[y + 1];
      }
    const uint32_t i = atomicAdd(&a.claim[x], 1u);
    if (i < (uint32_t)(x1 - x0)) {
      q = x;
      return (uint32_t)x0 + i;
    }
  }
  return end;
}

// The next work item as thread 0 learns it while the current one runs: the claim is issued
// when the item starts, and resolved once the epilogue has staged the tile, where the item
// word and the tile row are loaded too; the next item then starts with its descriptor at hand.
struct NextItem {
  uint32_t q;       // queue claimed from
  uint32_t ticket;  // the claim's position in queue q (in flight until resolved)
  int32_t q0, q1;   // queue q's bounds
  uint32_t pos;     // position of the next item in a.items, or end
  uint32_t item;
  TileRow tr;
  bool done;        // pos, item and tr are known
};

__device__ __forceinline__ void next_claim(const ProducerArgs& a, NextItem& n) {
  n.ticket = atomicAdd(&a.claim[n.q], 1u);
  n.q0 = a.queue[n.q];
  n.q1 = a.queue[n.q + 1];
  n.done = false;
}

__device__ __forceinline__ uint32_t item_tile_row(uint32_t item) {
  return (item >> kItemRowShift) & (uint32_t)(kMaxTileRows - 1);
}

// Resolves the claim (the other queues in turn if queue q ran dry) and loads the descriptor.
// Thread 0 runs this while the epilogue's stores are in flight: the item word and the tile row
// come through the scalar cache at a wave-uniform address, so the wait for them is not a wait
// for those stores.
__device__ __forceinline__ void next_resolve(const ProducerArgs& a, NextItem& n, uint32_t end) {
  if (n.done) return;
  if (n.ticket < (uint32_t)(n.q1 - n.q0)) {
    n.pos = (uint32_t)n.q0 + n.ticket;
  } else {
    n.pos = claim_item(a, n.q, end, false);  // queue q ran dry: any queue that has items
  }
  n.pos = __builtin_amdgcn_readfirstlane(n.pos);  // thread 0's value: one lane is active
  if (n.pos < end) {
    n.item = load_scalar(a.items + n.pos);
    const int32_t* w = (const int32_t*)(a.tile_rows + item_tile_row(n.item));
    n.tr.expert = load_scalar(w + 0);
    n.tr.lrow0 = load_scalar(w + 1);
    n.tr.nvalid = load_scalar(w + 2);
    n.tr.has_remote = load_scalar(w + 3);
    n.tr.split = load_scalar(w + 4);
    n.tr.part_base = load_scalar(w + 5);
  }
  n.done = true;
}

// Thread 0 hands the next item over through the shared words (the ring is idle).
__device__ __forceinline__ void next_publish(const ProducerArgs& a, NextItem& n, uint32_t end, uint32_t* words) {
  next_resolve(a, n, end);
  words[kWordPos] = n.pos;
  if (n.pos < end) {
    words[kWordItem] = n.item;
    words[kWordTileRow + 0] = (uint32_t)n.tr.expert;
    words[kWordTileRow + 1] = (uint32_t)n.tr.lrow0;
    words[kWordTileRow + 2] = (uint32_t)n.tr.nvalid;
    words[kWordTileRow + 3] = (uint32_t)n.tr.has_remote;
    words[kWordTileRow + 4] = (uint32_t)n.tr.split;
    words[kWordTileRow + 5] = (uint32_t)n.tr.part_base;
  }
}

// Every thread reads the published item (uniform values, kept in scalar registers).
__device__ __forceinline__ uint32_t read_item(const uint32_t* words, uint32_t& item, TileRow& tr) {
  const uint32_t pos = __builtin_amdgcn_readfirstlane(words[kWordPos]);
  item = __builtin_amdgcn_readfirstlane(words[kWordItem]);
  tr.expert = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 0]);
  tr.lrow0 = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 1]);
  tr.nvalid = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 2]);
  tr.has_remote = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 3]);
  tr.split = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 4]);
  tr.part_base = __builtin_amdgcn_readfirstlane((int)words[kWordTileRow + 5]);
  return pos;
}

// Persistent producer: every workgroup claims items from this launch's queues until they are
// empty.  Nothing inside waits on another workgroup, so progress never depends on which
// workgroups are resident.
template <bool down, int kSplit>
__global__ __launch_bounds__(kProducerThreads, 1) void producer_kernel(ProducerArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsBytes];
  uint32_t* words = (uint32_t*)(lds + kSharedWords);
  const int tid = threadIdx.x;
  // Where consumer waves share a SIMD with this wave (shared CUs), the producer's instructions
  // issue first: its workgroups are the stage's critical path, the consumer's copies are not.
  __builtin_amdgcn_s_setprio(3);
  // The init kernel has finished (it precedes this launch in the stream): release the consumer.
  if (!down && a.go_ctr && blockIdx.x == 0 && tid == 0)
    __hip_atomic_store(&a.go_ctr->go, a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t end = (uint32_t)a.queue[kXcds];
  const uint64_t t_start = ticks();
  const uint64_t c_start = clock64();
  NextItem nx;  // meaningful in thread 0, which does the claiming
  if (tid == 0) {
    nx.q = xcc_id();
    nx.pos = claim_item(a, nx.q, end, true);
    if (nx.pos < end) {
      atomicAdd(a.active, 1u);
      nx.item = a.items[nx.pos];
      nx.tr = a.tile_rows[item_tile_row(nx.item)];
    }
    nx.done = true;
    next_publish(a, nx, end, words);
  }
  __syncthreads();
  uint32_t item;
  TileRow tr;
  uint32_t cur = read_item(words, item, tr);
  int32_t n_items = 0;
  while (cur < end) {
    ++n_items;
    __syncthreads();  // every wave has read the words before the operand ring overwrites them
    // Thread 0 claims the next item two K steps before this one ends, late enough that a
    // workgroup slowed down (by consumer waves beside it) does not hold a claim on an item that
    // another one could start sooner, and early enough that the claim has returned by the
    // epilogue, where the item's descriptor is fetched; it is passed on through LDS at the end.
    auto late = [&]() {
      if (tid == 0) next_claim(a, nx);
    };
    auto hook = [&]() {
      if (tid == 0) next_resolve(a, nx, end);
    };
    if constexpr (kSplit < 0) {
      // Split per tile row: whole tiles take the plain epilogue, split rows the part path.
      if (tr.split == 1)
        producer_item<down, 1>(a, item, tr, lds, words, late, hook);
      else
        producer_item<down, 0>(a, item, tr, lds, words, late, hook);
    } else {
      producer_item<down, kSplit>(a, item, tr, lds, words, late, hook);
    }
    if (tid == 0) next_publish(a, nx, end, words);
    __syncthreads();
    cur = read_item(words, item, tr);
  }
  if (a.wg_rec && tid == 0) {  // timestamped runs: where and when this workgroup ran
    // The last item is done (a signalled down item has also waited for its stores).
    const uint64_t t_end = ticks();
    const uint64_t c_end = clock64();
    WgRecord r;
    r.hw_id = hw_id();
    r.xcc_id = xcc_id();
    r.launch = down ? 1 : 0;
    r.items = n_items;
    r.t_start = t_start;
    r.t_end = t_end;
    r.cycles = c_end - c_start;
    a.wg_rec[blockIdx.x] = r;
    if (down)
      __hip_atomic_fetch_max(&a.ctr->prod_t1, t_end, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      __hip_atomic_fetch_min(&a.ctr->prod_t0, t_start, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------------------
// Tail: the split tile rows of a kModeDeferTail down launch.  Their parts only stored fp32
// partials; here each workgroup pass takes one of a tile's 64 accumulator blocks, issues the
// loads of all its parts at once, adds them in part order from part 0 -- exactly the sums the
// last-arriving part would form -- and stores those outputs where the down epilogue would (Y
// at device scope, or the local receive buffer).  The last of a tile's 64 passes raises its
// flag.  Thread tid takes the positions producer thread tid held, so its loads are the 8-byte
// words that thread stored.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kProducerThreads) void tail_kernel(TailArgs ta) {
  const ProducerArgs& a = ta.p;
  __builtin_amdgcn_s_setprio(3);  // ahead of consumer waves on shared CUs, like the producer
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1, lr = lane & 31, lk = lane >> 5;
  const int dpr = a.down_per_row;
  const int64_t H = a.H;
  constexpr int kBlocks = 64;
  const int64_t n_pass = (int64_t)*ta.n_split_rows * dpr * kBlocks;
  const bool direct = (a.mode & kModeLocalDirect) != 0;
  const bool signal = (a.mode & kModeSignal) != 0;
  const bool direct_all = (a.mode & kModeDirectAll) != 0;
  constexpr int kPartU64 = kProducerThreads * 128;
  // The parts were stored by the previous launch at the coherence point; the launch's own
  // acquire makes them visible, so no fence (an L2 invalidate per workgroup) is needed here.
  for (int64_t pr = blockIdx.x; pr < n_pass; pr += gridDim.x) {
    const int t = ta.tail_rows[pr / (dpr * kBlocks)];
    const int col = (int)(pr / kBlocks % dpr), b = (int)(pr % kBlocks);
    const TileRow tr = a.tile_rows[t];
    const int S = tr.split;
    const uint64_t* src = (const uint64_t*)a.partials + ((size_t)tr.part_base + (size_t)col * S) * kPartU64 +
                          (2 * b) * kProducerThreads + tid;
    // Every part's two words in flight together (a part past the count re-reads the last one
    // and is not added).
    uint64_t lo[kMaxSplitK], hi[kMaxSplitK];
#pragma unroll
    for (int p = 0; p < kMaxSplitK; ++p) {
      const size_t o = (size_t)min(p, S - 1) * kPartU64;
      lo[p] = src[o];
      hi[p] = src[o + kProducerThreads];
    }
    float s0 = __uint_as_float((uint32_t)lo[0]), s1 = __uint_as_float((uint32_t)(lo[0] >> 32));
    float s2 = __uint_as_float((uint32_t)hi[0]), s3 = __uint_as_float((uint32_t)(hi[0] >> 32));
#pragma unroll
    for (int p = 1; p < kMaxSplitK; ++p)
      if (p < S) {
        s0 += __uint_as_float((uint32_t)lo[p]);
        s1 += __uint_as_float((uint32_t)(lo[p] >> 32));
        s2 += __uint_as_float((uint32_t)hi[p]);
        s3 += __uint_as_float((uint32_t)(hi[p] >> 32));
      }
    const int i = b >> 4, j = (b >> 2) & 3, q = b & 3;
    const int m = wm * 128 + j * 32 + lr;
    const int n = col * kDownTileN + wn * 128 + i * 32 + 8 * q + 4 * lk;
    const int lrow = tr.lrow0 + m;
    const int rank = a.row_rank[lrow];
    if (rank >= 0 && n < H) {
      const uint64_t v = (uint64_t)pack_bf16x2(s0, s1) | ((uint64_t)pack_bf16x2(s2, s3) << 32);
      if (direct_all || (direct && rank == a.self_rank)) {
        *(__attribute__((address_space(1))) uint64_t*)(a.ret[rank] + (int64_t)a.row_slot[lrow] * H + n) = v;
        count_words(a.wcount, lrow, 1);
      } else if (signal)
        store8_device(a.y + (int64_t)lrow * H + n, v);
      else
        *(__attribute__((address_space(1))) uint64_t*)(a.y + (int64_t)lrow * H + n) = v;
    }
    if (signal && (tr.has_remote || !direct)) {
      // Every wave's stores have completed before the pass counts itself in; the pass that
      // completes the tile raises the flag.
      wait_vm_and_barrier<0>();
      if (tid == 0) {
        const int tile = t * dpr + col;
        const uint32_t prev =
            __hip_atomic_fetch_add(&a.arrivals[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (prev + 1 == (uint32_t)kBlocks) {
          if (a.tile_ready) a.tile_ready[tile] = ticks();
          __hip_atomic_store(&a.flags[tile], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }
  if (a.wg_rec && n_pass > 0) {  // timestamped runs: the producer ends with its last tail pass
    wait_vm_and_barrier<0>();
    if (tid == 0) __hip_atomic_fetch_max(&a.ctr->prod_t1, ticks(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------------------
// Consumer: every wave works alone.  It claims a copy unit -- one of a segment's 2^shift equal
// parts, in the segments' ready order -- polls the segment's flags (one flag per lane; all
// must show the current epoch), then copies its part with 16-byte loads and stores.  The
// kernel uses no LDS, so in a shared-CU run its workgroups never keep a producer workgroup
// (which takes all of LDS) off a compute unit.
//
// kOwn = false (beside the producer): at most 56 VGPRs per wave, so two consumer waves fit
// beside a producer wave on a SIMD.  A copying wave slows the producer workgroup on its compute
// unit, so the launch spreads about 256 waves over the split's compute units (one per compute
// unit on a wide split, eight on a narrow one), and a wave that finds its SIMD or its compute unit
// already holding its share exits at once: consumer waves that happened to pile onto one compute
// unit before the producer arrived never keep a producer workgroup off it, nor crowd its memory
// path.  The first tickets are dealt transposed, so the waves of one workgroup, which claim
// together, take parts of different segments.  kOwn = true (compute units of its own): up to 128
// VGPRs, about three times the data in flight per wave.
// ---------------------------------------------------------------------------

// Copies n 16-byte vectors from src to dst, kU per lane per chunk, with two register buffers in
// turn so one chunk's loads are in flight while the other's stores issue.
//
// The staged rows are read with agent-scope coherent buffer loads (cache policy sc1): each load
// sees what the producer stored at the coherence point, whichever XCD it ran on, so the copy needs
// no acquire fence after the flag poll.  On gfx950 an agent-scope acquire invalidates the XCD's
// whole L2, which would throw away the operand panels the producer workgroups on that XCD keep
// there (one invalidation per copy unit while the down launch runs).  No streaming (nt) hint: rows
// the producer has just written are often still in the memory-side cache, and an nt load of them
// went slower (a 100 MB copy by 10-30 %) with no gain for the producer beside it.  The source run
// is below 4 GiB (the handle's staged output is), so 32-bit buffer offsets reach all of it.
constexpr int kLoadAgent = 16;  // buffer-load cache policy: sc1 (agent scope)

template <int kU>
__device__ __forceinline__ void copy_vectors(const void* src, g_u32x4* __restrict__ dst, int64_t n, int lane) {
  constexpr int64_t kStep = (int64_t)kU * 64;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(src), 0, (int)(uint32_t)min<int64_t>(n * 16, INT_MAX), kBufferRsrcWord3);
  auto ld = [&](int64_t i) { return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(i * 16), 0, kLoadAgent); };
  const int64_t nfull = n / kStep;
  u32x4 a[kU], b[kU];
  auto load = [&](u32x4 (&r)[kU], int64_t c) {
#pragma unroll
    for (int u = 0; u < kU; ++u) r[u] = ld(c * kStep + lane + u * 64);
  };
  auto store = [&](const u32x4 (&r)[kU], int64_t c) {
#pragma unroll
    for (int u = 0; u < kU; ++u) __builtin_nontemporal_store(r[u], dst + (c * kStep + lane + u * 64));
  };
  if (nfull > 0) {
    load(a, 0);
    int64_t c = 0;
    for (; c + 1 < nfull; c += 2) {
      load(b, c + 1);
      store(a, c);
      if (c + 2 < nfull) load(a, c + 2);
      store(b, c + 1);
    }
    if (c < nfull) store(a, c);
  }
  for (int64_t i = nfull * kStep + lane; i < n; i += 64) dst[i] = ld(i);
}

// Plan words read at agent scope (sc1): coherent with what the run's upload or the device planner
// wrote, whichever XCD cached an older plan, so the consumer needs no acquire fence (on gfx950 an
// agent-scope acquire invalidates the XCD's whole L2, under the producer's feet).
__device__ __forceinline__ int32_t ld_agent(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ Segment load_segment(const Segment* p) {
  Segment sg;
  sg.dst_rank = ld_agent(&p->dst_rank);
  sg.rows = ld_agent(&p->rows);
  sg.y_row0 = ld_agent(&p->y_row0);
  sg.slot0 = ld_agent(&p->slot0);
  sg.flag_begin = ld_agent(&p->flag_begin);
  sg.flag_count = ld_agent(&p->flag_count);
  sg.ready_pos = ld_agent(&p->ready_pos);
  sg.npieces = ld_agent(&p->npieces);
  return sg;
}

// The receive buffer of rank r, read from the run's pointer table at agent scope.
__device__ __forceinline__ uint16_t* ret_buffer(uint16_t* const* table, int r) {
  const uint64_t v = __hip_atomic_load((const uint64_t*)(table + r), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return (uint16_t*)(uintptr_t)v;
}

// The units of a run: segments in ready order, the first n_early (ready before the last round
// of the down queues) cut into 2^early_shift units each, the others into 2^late_shift.
struct UnitCounts {
  int32_t n_early;
  uint32_t early_units, n_units;
};

__device__ __forceinline__ UnitCounts unit_counts(const ConsumerArgs& a) {
  const int32_t n_segs = ld_agent(a.n_segs);
  // Segments are in ready order: the first late one by binary search (uniform loads).
  const int32_t late_from = ld_agent(a.down_qmax) - kLatePositions;
  UnitCounts u;
  u.n_early = 0;
  for (int32_t hi = n_segs; u.n_early < hi;) {
    const int32_t mid = (u.n_early + hi) >> 1;
    if (ld_agent(&a.segs[mid].ready_pos) < late_from)
      u.n_early = mid + 1;
    else
      hi = mid;
  }
  u.early_units = (uint32_t)u.n_early << a.early_shift;
  u.n_units = u.early_units + ((uint32_t)(n_segs - u.n_early) << a.late_shift);
  return u;
}

// MOE_WRITE_COUNTS: a copied run of vectors [i0, i1) of a segment whose rows start at logical row
// y_row0 counts, for each row it touches, the 8-byte words it wrote there.
__device__ __forceinline__ void count_copy(uint32_t* wcount, int32_t y_row0, uint32_t per_row, uint32_t i0,
                                           uint32_t i1, int lane) {
  if (!wcount || i1 <= i0) return;
  for (uint32_t r = i0 / per_row + (uint32_t)lane; r <= (i1 - 1) / per_row; r += 64) {
    const uint32_t a = max(i0, r * per_row), b = min(i1, (r + 1) * per_row);
    count_words(wcount, (int64_t)y_row0 + r, 2 * (b - a));
  }
}

// Copies unit `unit` with no flag wait (its rows are known complete).
template <bool kOwn, bool kCount>
__device__ __forceinline__ void copy_unit(const ConsumerArgs& a, const UnitCounts& uc, uint32_t unit, int lane) {
  if (unit >= uc.n_units) return;
  const bool early = unit < uc.early_units;
  const uint32_t u = early ? unit : unit - uc.early_units;
  const int32_t shift = early ? a.early_shift : a.late_shift;
  const int32_t s = (early ? 0 : uc.n_early) + (int32_t)(u >> shift);
  const int32_t part = (int32_t)(u & ((1u << shift) - 1));
  const Segment sg = load_segment(a.segs + s);
  const int64_t n16 = (int64_t)sg.rows * a.H / 8;
  const int64_t i0 = (n16 * part) >> shift, i1 = (n16 * (part + 1)) >> shift;
  const u32x4* src = (const u32x4*)(a.y + (int64_t)sg.y_row0 * a.H) + i0;
  g_u32x4* dst = (g_u32x4*)(ret_buffer(a.ret, sg.dst_rank) + (int64_t)sg.slot0 * a.H) + i0;
  copy_vectors<kOwn ? kCopyUnrollOwn : kCopyUnroll>(src, dst, i1 - i0, lane);
  if constexpr (kCount) count_copy(a.wcount, sg.y_row0, (uint32_t)(a.H / 8), (uint32_t)i0, (uint32_t)i1, lane);
}

// The ticket loop of one wave: claim a copy unit, wait for its segment's flags, copy its part.
// The first n_waves tickets are dealt transposed over the waves of the launch that map_grid and
// map_wpg describe (ticket w_per_wg * b + w to unit w * map_grid + b), so the waves of one
// workgroup, which claim together, take parts of different segments; later tickets are units in
// order.
template <bool kOwn, bool kCount>
__device__ __forceinline__ void consume_units(const ConsumerArgs& a, const UnitCounts& uc, int lane) {
  const uint32_t wpg = a.map_wpg ? a.map_wpg : blockDim.x >> 6;
  const uint32_t map_grid = a.map_grid ? a.map_grid : gridDim.x;
  const uint32_t n_waves = map_grid * wpg;
  const int32_t n_early = uc.n_early;
  const int32_t early_shift = a.early_shift, late_shift = a.late_shift;
  const uint32_t early_units = uc.early_units, n_units = uc.n_units;
  const uint32_t last_ticket = max(n_waves, n_units);
  uint32_t polls = 0;
  uint64_t waited = 0;
  for (;;) {
    uint32_t t = 0;
    if (lane == 0) t = atomicAdd(&a.ctr->seg_next, 1u);
    t = __builtin_amdgcn_readfirstlane(t);  // every lane is active here
    if (t >= last_ticket) break;
    const uint32_t unit = t < n_waves ? (t % wpg) * map_grid + t / wpg : t;
    if (unit >= n_units) continue;
    const bool early = unit < early_units;
    const uint32_t u = early ? unit : unit - early_units;
    const int32_t shift = early ? early_shift : late_shift;
    const int32_t s = (early ? 0 : n_early) + (int32_t)(u >> shift);
    const int32_t part = (int32_t)(u & ((1u << shift) - 1));
    const Segment sg = load_segment(a.segs + s);
    const uint64_t t0 = ticks();
    bool expired = false;
    uint32_t backoff = 1;
    // The drain follows the producer and its tail kernel in their stream, so every row it copies
    // is complete: it does not poll.
    const int flag_count = (kOwn && a.role == kRoleDrain) ? 0 : sg.flag_count;
    for (int base = 0; base < flag_count && !expired; base += 64) {
      const bool mine = base + lane < flag_count;
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
        // Exponential backoff: a wave that waits through the whole gate/up launch settles at
        // one poll every 2.5 us or so, instead of flooding L2 with flag loads.
        for (uint32_t i = 0; i < backoff; ++i) __builtin_amdgcn_s_sleep(kPollSleep);
        backoff = backoff < kPollBackoffMax ? 2 * backoff : kPollBackoffMax;
      }
    }
    // No acquire: the copy's loads are agent-scope coherent (see copy_vectors).
    const uint64_t t_ready = ticks();
    waited += t_ready - t0;
    if (expired) {
      // The wave gives up (the producer is not making progress beside it) and hands the unit to
      // the drain launch, which copies it after the producer: the run is slow but complete.
      if (lane == 0) {
        __hip_atomic_fetch_add(&a.ctr->timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_or(&a.ctr->timeout_where, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_min(&a.ctr->timeout_seg, (uint32_t)s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (a.abandoned) {
          const uint32_t k = __hip_atomic_fetch_add(&a.ctr->n_abandoned, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (k < a.abandoned_cap)
            __hip_atomic_store(&a.abandoned[k], unit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      break;
    }
    // The segment is contiguous on both sides: this wave's part is a flat run of 16-byte vectors.
    const int64_t n16 = (int64_t)sg.rows * a.H / 8;
    const int64_t i0 = (n16 * part) >> shift, i1 = (n16 * (part + 1)) >> shift;
    const u32x4* src = (const u32x4*)(a.y + (int64_t)sg.y_row0 * a.H) + i0;  // wave-uniform
    g_u32x4* dst = (g_u32x4*)(ret_buffer(a.ret, sg.dst_rank) + (int64_t)sg.slot0 * a.H) + i0;
    copy_vectors<kOwn ? kCopyUnrollOwn : kCopyUnroll>(src, dst, i1 - i0, lane);
    if constexpr (kCount) count_copy(a.wcount, sg.y_row0, (uint32_t)(a.H / 8), (uint32_t)i0, (uint32_t)i1, lane);
    if (a.rec && unit < a.rec_cap) {
      // Timestamped runs: the unit ends when its stores have completed.
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      const uint64_t t_done = ticks();
      // One dword of the record per lane: a whole record in lane 0 would hold twelve
      // registers at once, past this variant's budget.
      constexpr int kWords = (int)(sizeof(CopyRecord) / 4);
      if (lane < kWords) {
        const uint32_t source = kOwn && a.role == kRoleDrain ? 1u : 0u;  // the drain is a kOwn launch
        uint32_t w = 0;
        switch (lane) {
          case 0: w = (uint32_t)s; break;
          case 1: w = (uint32_t)part; break;
          case 2: w = hw_id(); break;
          case 3: w = xcc_id(); break;
          case 4: w = (uint32_t)t0; break;
          case 5: w = (uint32_t)(t0 >> 32); break;
          case 6: w = (uint32_t)t_ready; break;
          case 7: w = (uint32_t)(t_ready >> 32); break;
          case 8: w = (uint32_t)t_done; break;
          case 9: w = (uint32_t)(t_done >> 32); break;
          case 10: w = source; break;
          default: break;
        }
        reinterpret_cast<uint32_t*>(a.rec + unit)[lane] = w;
      }
    }
  }
  if (lane == 0 && (polls || waited)) {
    atomicAdd((unsigned long long*)&a.ctr->poll_iters, (unsigned long long)polls);
    atomicAdd((unsigned long long*)&a.ctr->wait_ticks, (unsigned long long)waited);
  }
}

// A counted consumer wave's exit: its copies are complete and written back from its XCD's L2
// before the count rises, so the drain launch's end covers them.
__device__ __forceinline__ void count_exit(const ConsumerArgs& a, int lane) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  if (lane == 0) __hip_atomic_fetch_add(&a.ctr->cons_exit, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// kCount: the MOE_WRITE_COUNTS variant, which also counts what it writes (outside the register budget).
template <bool kOwn, bool kCount>
__global__ __launch_bounds__(kConsumerThreads, kOwn ? kConsumerOwnMinWaves : kConsumerMinWaves)
void consumer_kernel(ConsumerArgs a) {
  const int lane = threadIdx.x & 63;
  if (a.wait_go) {
    // Launched with no stream dependency on this run's reset: wait until the reset has
    // published the run's epoch.  If that takes past the watchdog (the caller's stream still
    // busy with earlier work), leave without claiming anything: the drain launch, which
    // follows the producer in its stream, copies every unit, so this costs only the overlap.
    const uint64_t t0 = ticks();
    uint32_t backoff = 1;
    bool go = true;
    while (__hip_atomic_load(&a.ctr->go, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != a.epoch) {
      if (ticks() - t0 > a.watchdog_ticks) {
        go = false;
        break;
      }
      for (uint32_t i = 0; i < backoff; ++i) __builtin_amdgcn_s_sleep(kPollSleep);
      backoff = backoff < kPollBackoffMax ? 2 * backoff : kPollBackoffMax;
    }
    // No acquire fence: every plan word, flag and staged row the consumer reads afterwards is read
    // at agent scope.
    if (!go) {
      if (a.role == kRoleCounted) count_exit(a, lane);
      return;
    }
  }
  if (!kOwn && a.simd_waves) {
    // hw_id: SIMD [5:4], compute unit [11:8], shader array [12], shader engine [15:13].
    // A wave past either limit leaves at once.
    uint32_t over = 0;
    if (lane == 0) {
      const uint32_t h = hw_id();
      const uint32_t key = ((((h >> 13) & 7u) * 2 + ((h >> 12) & 1u)) * 16 + ((h >> 8) & 15u)) * 4 + ((h >> 4) & 3u);
      const uint32_t x = xcc_id();
      over = atomicAdd(&a.simd_waves[x * kSimdKeys + key], 1u) >= (uint32_t)kMaxConsumerWavesPerSimd;
      if (!over && a.max_waves_cu)
        over = atomicAdd(&a.simd_waves[kXcds * kSimdKeys + x * kCuKeys + (key >> 2)], 1u) >= a.max_waves_cu;
    }
    if (__builtin_amdgcn_readfirstlane(over)) {
      if (a.role == kRoleCounted) count_exit(a, lane);
      return;
    }
  }
  UnitCounts uc;
  bool known = false;
  if (kOwn && a.role == kRoleDrain) {
    // The consumer has published the unit counts, so the drain skips the unit map (a chain of
    // dependent loads).
    const uint64_t pub = __hip_atomic_load(&a.ctr->units_pub, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (pub != 0) {
      uc.n_units = (uint32_t)(pub >> 32);
      uc.early_units = (uint32_t)pub;
      uc.n_early = (int32_t)(uc.early_units >> a.early_shift);
      known = true;
    }
  }
  if (!known) {
    uc = unit_counts(a);
    if (!(kOwn && a.role == kRoleDrain) && blockIdx.x == 0 && threadIdx.x == 0) {
      // Published at agent scope: the drain launch reads them from other XCDs.
      __hip_atomic_store(&a.ctr->n_units, uc.n_units, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctr->units_pub, ((uint64_t)uc.n_units << 32) | uc.early_units, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  bool tickets = true;
  if (known) {
    // Usually the consumer has taken every ticket, and the drain skips the ticket loop.
    const uint32_t next = __hip_atomic_load(&a.ctr->seg_next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t wpg = a.map_wpg ? a.map_wpg : blockDim.x >> 6;
    tickets = next < max(a.map_grid * wpg, uc.n_units);
  }
  if (tickets) consume_units<kOwn, kCount>(a, uc, lane);
  if (a.role == kRoleCounted) {
    count_exit(a, lane);
  } else if (kOwn && a.role == kRoleDrain && blockIdx.x == 0 && threadIdx.x < 64) {
    // Every ticket is claimed; the consumer's waves still copying finish on their own (each
    // unit's flags are raised, the producer having ended), and waves not yet started find no
    // ticket left.  The wait is bounded like every flag wait.
    const uint64_t t0 = ticks();
    uint32_t backoff = 1;
    while (__hip_atomic_load(&a.ctr->cons_exit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < a.exit_waves) {
      if (ticks() - t0 > a.watchdog_ticks) {
        if (lane == 0) {
          __hip_atomic_fetch_add(&a.ctr->timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_fetch_or(&a.ctr->timeout_where, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        break;
      }
      for (uint32_t i = 0; i < backoff; ++i) __builtin_amdgcn_s_sleep(1);
      backoff = backoff < 8 ? 2 * backoff : 8;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    // Units a consumer wave abandoned when its flag wait expired: every consumer wave has exited,
    // so the list is complete, and the producer has finished, so the rows are.
    const uint32_t n_ab = min(__hip_atomic_load(&a.ctr->n_abandoned, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                              a.abandoned_cap);
    for (uint32_t k = 0; a.abandoned && k < n_ab; ++k)
      copy_unit<kOwn, kCount>(a, uc, __hip_atomic_load(&a.abandoned[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), lane);
  }
}

// ---------------------------------------------------------------------------
// Measurement aid: as many bytes as the consumer's segments hold, copied from the staged
// output into the first receive buffer by a plain grid-stride loop, 8 vectors in flight per
// lane -- what the same compute units reach on a flat copy of the same size, with no protocol.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kConsumerThreads) void plain_copy_kernel(ConsumerArgs a) {
  const int64_t stride = (int64_t)gridDim.x * kConsumerThreads;
  const int64_t n = a.plain_n16;
  const u32x4* src = (const u32x4*)a.y;
  g_u32x4* dst = (g_u32x4*)a.ret[0];
  constexpr int kU = 8;
  for (int64_t i = (int64_t)blockIdx.x * kConsumerThreads + threadIdx.x; i < n; i += kU * stride) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (i + u * stride < n) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (i + u * stride < n) dst[i + u * stride] = v[u];
  }
}

hipError_t launch_plain_copy(const ConsumerArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(plain_copy_kernel, dim3(grid), dim3(kConsumerThreads), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Baseline bulk return: every routed row of the staged output to its slot.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a) {
  const int64_t per_row = a.H / 8;
  const int64_t n_lrows = *a.n_lrows;
  for (int64_t r = blockIdx.x; r < n_lrows; r += gridDim.x) {
    const int rank = a.row_rank[r];
    if (rank < 0) continue;
    const u32x4* src = (const u32x4*)(a.y + r * a.H);
    g_u32x4* dst = (g_u32x4*)(a.ret[rank] + (int64_t)a.row_slot[r] * a.H);
    for (int64_t i = threadIdx.x; i < per_row; i += blockDim.x) dst[i] = src[i];
    if (threadIdx.x == 0) count_words(a.wcount, r, (uint32_t)(2 * per_row));
  }
}

__global__ __launch_bounds__(256) void init_kernel(InitArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i == 0) {
    for (int x = 0; x < kXcds; ++x) {
      a.ctr->gu_next[x] = 0;
      a.ctr->down_next[x] = 0;
    }
    a.ctr->seg_next = 0;
    a.ctr->gu_active = 0;
    a.ctr->down_active = 0;
    a.ctr->poll_iters = 0;
    a.ctr->wait_ticks = 0;
    a.ctr->n_units = 0;
    a.ctr->cons_exit = 0;
    a.ctr->units_pub = 0;
    a.ctr->prod_t0 = ~0ull;
    a.ctr->prod_t1 = 0;
    a.ctr->n_abandoned = 0;
    if (a.plan_hdr) {
      a.plan_hdr->status = 0;
      a.plan_hdr->bad_row = INT_MAX;
    }
  }
  if (a.fill_ones)
    for (int64_t j = i; j < a.n_fill_ones; j += stride) a.fill_ones[j] = ~0u;
  for (int64_t j = i; j < a.n_arrivals; j += stride) a.arrivals[j] = 0;
  if (a.wcount)
    for (int64_t j = i; j < a.n_wcount; j += stride) a.wcount[j] = 0;
  if (a.tile_ready)
    for (int64_t j = i; j < a.n_arrivals; j += stride) a.tile_ready[j] = 0;
  if (a.simd_waves)
    for (int64_t j = i; j < kWaveCounters; j += stride) a.simd_waves[j] = 0;
  // Published flags are stored as the producer raises them (relaxed, agent scope): a plain store
  // would sit in this XCD's L2, and the consumer's polls on other XCDs would not see it until the
  // line is written back.
  if (a.publish)
    for (int64_t j = i; j < a.n_publish; j += stride)
      __hip_atomic_store(&a.publish[j], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (a.poison) {
    const u32x4 nan = {0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};
    for (int64_t j = i; j < a.poison_elems / 8; j += stride) ((u32x4*)a.poison)[j] = nan;
  }
}

hipError_t launch_init(const InitArgs& a, hipStream_t s) {
  int grid = 64;
  if (a.poison || a.n_fill_ones > (1 << 18)) grid = 1024;
  hipLaunchKernelGGL(init_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_producer(const ProducerArgs& a, bool down, int grid, hipStream_t s) {
  const dim3 g(grid), b(kProducerThreads);
  if (!down)
    hipLaunchKernelGGL((producer_kernel<false, 1>), g, b, 0, s, a);
  else if (a.split_k == 0)
    hipLaunchKernelGGL((producer_kernel<true, -1>), g, b, 0, s, a);
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

__global__ void go_kernel(RunCounters* ctr, uint32_t epoch) {
  if (threadIdx.x == 0) __hip_atomic_store(&ctr->go, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_go(RunCounters* ctr, uint32_t epoch, hipStream_t s) {
  hipLaunchKernelGGL(go_kernel, dim3(1), dim3(64), 0, s, ctr, epoch);
  return hipGetLastError();
}

hipError_t launch_drain(const ConsumerArgs& a, int grid, hipStream_t s) {
  if (a.wcount)
    hipLaunchKernelGGL((consumer_kernel<true, true>), dim3(grid), dim3(kConsumerThreads), 0, s, a);
  else
    hipLaunchKernelGGL((consumer_kernel<true, false>), dim3(grid), dim3(kConsumerThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_consumer(const ConsumerArgs& a, bool own_cus, int grid, int threads, hipStream_t s) {
  if (threads <= 0 || threads > kConsumerThreads || threads % 64) return hipErrorInvalidValue;
  const dim3 g(grid), b(threads);
  if (own_cus && a.wcount)
    hipLaunchKernelGGL((consumer_kernel<true, true>), g, b, 0, s, a);
  else if (own_cus)
    hipLaunchKernelGGL((consumer_kernel<true, false>), g, b, 0, s, a);
  else if (a.wcount)
    hipLaunchKernelGGL((consumer_kernel<false, true>), g, b, 0, s, a);
  else
    hipLaunchKernelGGL((consumer_kernel<false, false>), g, b, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tail(const TailArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(tail_kernel, dim3(grid), dim3(kProducerThreads), 0, s, a);
  return hipGetLastError();
}

// Writes the GPU's 100 MHz real-time counter to *dst (pinned host memory) when the stream
// reaches it: the adaptive split times its candidates with a pair of these, not with timing
// events recorded inside the runs it measures.
__global__ void stamp_kernel(uint64_t* dst) {
  if (threadIdx.x == 0) {
    *dst = ticks();
    __threadfence_system();
  }
}

hipError_t launch_stamp(uint64_t* dst, hipStream_t s) {
  hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, s, dst);
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
