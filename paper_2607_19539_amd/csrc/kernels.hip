// kernels.hip -- gfx950 (MI355X, CDNA4) kernels of the MoE expert stage.
//
//  * producer: persistent rank-wide grouped gated-FFN GEMM (paper Section
//    3.3.1).  One work queue covers every local expert; an item is one
//    256x256 output tile of either the fused gate/up projection (128 ffn
//    features, both projections, SiLU-gated in the epilogue) or the down
//    projection.  Each finished down tile of a tile row that needs a transfer
//    publishes a ready flag with an agent-scope release (the epilogue signal
//    of Section 3.3.1).
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

#include "kernels.hpp"

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Operand tile in LDS: 256 rows x 64 k (bf16) = 32 KiB, 128 bytes per row.  The
// 16-byte chunk index is XOR-swizzled with the row so that the 32 rows read by
// one MFMA operand load spread over all banks (conflict-free for 8-lane and
// 16-lane bank phases alike).
constexpr int kRowBytes = kTileK * 2;
constexpr int kOperandBytes = kTileM * kRowBytes;   // 32 KiB
constexpr int kStageBytes = 2 * kOperandBytes;      // weight tile + token tile
constexpr int kLdsBytes = 2 * kStageBytes;          // double buffered: 128 KiB

__device__ __forceinline__ uint32_t swz(uint32_t row) { return (row & 7u) ^ ((row >> 3) & 1u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

__device__ __forceinline__ uint64_t ticks() { return wall_clock64(); }

// ---------------------------------------------------------------------------
// One 256x256 output tile: acc[i][j] holds D[n][m] for the wave's 128x128
// quadrant, n = wn*128 + i*32 + 8*(r/4) + 4*(lane/32) + r%4, m = wm*128 + j*32 + lane%32.
// wp[i] / xp[i] point at row (tid/8 + 32 i) of the weight / token operand, already
// offset by this thread's 16-byte chunk (tid%8).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void tile_mma(uint8_t* __restrict__ lds, const uint16_t* const (&wp)[8],
                                         const uint16_t* const (&xp)[8], int K, f32x16 (&acc)[4][4]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const int r0 = tid >> 3, c = tid & 7;
  const uint32_t st_off = (uint32_t)r0 * kRowBytes + ((c ^ swz(r0)) << 4);
  const int lr = lane & 31, lk = lane >> 5;
  const uint32_t lsw = swz(lr);
  const uint32_t a_row = (uint32_t)(wn * 128 + lr) * kRowBytes;
  const uint32_t b_row = (uint32_t)(wm * 128 + lr) * kRowBytes;

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  u32x4 rw[8], rx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    rw[i] = *(const u32x4*)(wp[i]);
    rx[i] = *(const u32x4*)(xp[i]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    *(u32x4*)(lds + st_off + i * 4096) = rw[i];
    *(u32x4*)(lds + kOperandBytes + st_off + i * 4096) = rx[i];
  }
  __syncthreads();

  const int nk = K / kTileK;
  for (int ks = 0; ks < nk; ++ks) {
    uint8_t* cur = lds + (ks & 1) * kStageBytes;
    uint8_t* nxt = lds + ((ks + 1) & 1) * kStageBytes;
    const bool more = ks + 1 < nk;
    if (more) {
      const int koff = (ks + 1) * kTileK;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        rw[i] = *(const u32x4*)(wp[i] + koff);
        rx[i] = *(const u32x4*)(xp[i] + koff);
      }
    }
#pragma unroll
    for (int kk = 0; kk < kTileK / 16; ++kk) {
      const uint32_t coff = ((uint32_t)(2 * kk + lk) ^ lsw) << 4;
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = *(const bf16x8*)(cur + a_row + i * 32 * kRowBytes + coff);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = *(const bf16x8*)(cur + kOperandBytes + b_row + j * 32 * kRowBytes + coff);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        *(u32x4*)(nxt + st_off + i * 4096) = rw[i];
        *(u32x4*)(nxt + kOperandBytes + st_off + i * 4096) = rx[i];
      }
    }
    __syncthreads();
  }
}

__device__ void producer_item(const ProducerArgs& a, uint32_t item, uint8_t* lds, uint64_t& wait_acc) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const int lr = lane & 31, lk = lane >> 5;
  const bool down = (item & kItemDown) != 0;
  const int t = (int)((item >> kItemRowShift) & (uint32_t)(kMaxTileRows - 1));
  const int col = (int)(item & kItemColMask);
  const TileRow tr = a.tile_rows[t];
  const int64_t H = a.H, F = a.F;
  const int e = tr.expert, lrow0 = tr.lrow0;
  const int r0 = tid >> 3, c = tid & 7;

  const uint16_t* wp[8];
  const uint16_t* xp[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int n = r0 + 32 * i;  // row of the weight operand tile
    if (!down) {
      // Rows 0..63 / 128..191 hold gate features, 64..127 / 192..255 the matching up
      // features, so each wave's quadrant holds gate and up of the same 64 features.
      const int half = n >> 7, w = n & 127;
      const int f = min(col * kGuTileF + half * 64 + (w & 63), (int)F - 1);
      wp[i] = (w < 64 ? a.w1 : a.w3) + ((int64_t)e * F + f) * H + c * 8;
      xp[i] = a.x + (int64_t)a.row_x[lrow0 + n] * H + c * 8;
    } else {
      const int hcol = min(col * kDownTileN + n, (int)H - 1);
      wp[i] = a.w2 + ((int64_t)e * H + hcol) * F + c * 8;
      xp[i] = a.hws + (int64_t)(lrow0 + n) * F + c * 8;
    }
  }

  if (down) {
    // Every gate/up tile of this tile row must have published its activation.
    __shared__ uint32_t s_timeout;
    if (tid == 0) {
      s_timeout = 0;
      const uint64_t t0 = ticks();
      while (__hip_atomic_load(&a.gu_done[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
             (uint32_t)a.gu_per_row) {
        if (ticks() - t0 > a.watchdog_ticks) {
          s_timeout = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      wait_acc += ticks() - t0;
    }
    __syncthreads();
    if (s_timeout) {
      if (tid == 0) {
        __hip_atomic_fetch_add(&a.ctr->timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_or(&a.ctr->timeout_where, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      return;
    }
  }

  f32x16 acc[4][4];
  tile_mma(lds, wp, xp, down ? (int)F : (int)H, acc);

  if (!down) {
    const int f_base = col * kGuTileF + wn * 64;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int lrow = lrow0 + wm * 128 + j * 32 + lr;
      if (a.row_rank[lrow] < 0) continue;  // padding rows are never read back
      uint16_t* dst = a.hws + (int64_t)lrow * F;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int f = f_base + i * 32 + 8 * q + 4 * lk;
          if (f < F) {
            const f32x16& g = acc[i][j];
            const f32x16& u = acc[i + 2][j];
            uint2 v;
            v.x = pack_bf16x2(silu_mul(g[4 * q + 0], u[4 * q + 0]), silu_mul(g[4 * q + 1], u[4 * q + 1]));
            v.y = pack_bf16x2(silu_mul(g[4 * q + 2], u[4 * q + 2]), silu_mul(g[4 * q + 3], u[4 * q + 3]));
            *(uint2*)(dst + f) = v;
          }
        }
    }
    __syncthreads();
    if (tid == 0)
      __hip_atomic_fetch_add(&a.gu_done[t], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    const int n_base = col * kDownTileN + wn * 128;
    const bool direct = (a.mode & kModeLocalDirect) != 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int lrow = lrow0 + wm * 128 + j * 32 + lr;
      const int rank = a.row_rank[lrow];
      if (rank < 0) continue;
      uint16_t* dst = (direct && rank == a.self_rank)
                          ? a.ret[rank] + (int64_t)a.row_slot[lrow] * H
                          : a.y + (int64_t)lrow * H;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int n = n_base + i * 32 + 8 * q + 4 * lk;
          if (n < H) {
            const f32x16& d = acc[i][j];
            uint2 v;
            v.x = pack_bf16x2(d[4 * q + 0], d[4 * q + 1]);
            v.y = pack_bf16x2(d[4 * q + 2], d[4 * q + 3]);
            *(uint2*)(dst + n) = v;
          }
        }
    }
    if ((a.mode & kModeSignal) && (tr.has_remote || !direct)) {
      __syncthreads();
      if (tid == 0)
        __hip_atomic_store(&a.flags[t * a.down_per_row + col], a.epoch, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__global__ __launch_bounds__(kProducerThreads, 1) void producer_kernel(ProducerArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsBytes];
  __shared__ uint32_t s_next;
  const int tid = threadIdx.x;
  uint64_t wait_acc = 0;
  if (tid == 0) s_next = atomicAdd(&a.ctr->work_next, 1u);
  __syncthreads();
  uint32_t cur = s_next;
  while (cur < (uint32_t)a.n_items) {
    __syncthreads();
    // Claim the next item now; its index is read after this one finishes.  Items are
    // claimed in schedule order, so a tile only ever waits on tiles claimed earlier.
    if (tid == 0) s_next = atomicAdd(&a.ctr->work_next, 1u);
    producer_item(a, a.items[cur], lds, wait_acc);
    __syncthreads();
    cur = s_next;
  }
  if (tid == 0 && wait_acc) atomicAdd((unsigned long long*)&a.ctr->producer_wait_ticks, (unsigned long long)wait_acc);
}

// ---------------------------------------------------------------------------
// Consumer: claim segments in ready order; wave 0 polls the segment's flags
// (one flag per lane, all lanes must read the current epoch), then the whole
// workgroup copies rows * H bf16 with 16-byte loads and stores.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kConsumerThreads) void consumer_kernel(ConsumerArgs a) {
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
    const u32x4* src = (const u32x4*)(a.y + (int64_t)sg.y_row0 * a.H);
    u32x4* dst = (u32x4*)(a.ret[sg.dst_rank] + (int64_t)sg.slot0 * a.H);
    const int64_t n16 = (int64_t)sg.rows * a.H / 8;
    int64_t i = tid;
    for (; i + 3 * kConsumerThreads < n16; i += 4 * kConsumerThreads) {
      const u32x4 v0 = src[i], v1 = src[i + kConsumerThreads], v2 = src[i + 2 * kConsumerThreads],
                  v3 = src[i + 3 * kConsumerThreads];
      dst[i] = v0;
      dst[i + kConsumerThreads] = v1;
      dst[i + 2 * kConsumerThreads] = v2;
      dst[i + 3 * kConsumerThreads] = v3;
    }
    for (; i < n16; i += kConsumerThreads) dst[i] = src[i];
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
    u32x4* dst = (u32x4*)(a.ret[rank] + (int64_t)a.row_slot[r] * a.H);
    for (int64_t i = threadIdx.x; i < per_row; i += blockDim.x) dst[i] = src[i];
  }
}

__global__ __launch_bounds__(256) void init_kernel(InitArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (i == 0) {
    a.ctr->work_next = 0;
    a.ctr->seg_next = 0;
    a.ctr->poll_iters = 0;
    a.ctr->wait_ticks = 0;
    a.ctr->producer_wait_ticks = 0;
  }
  for (int64_t j = i; j < a.n_tile_rows; j += stride) a.gu_done[j] = 0;
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

hipError_t launch_producer(const ProducerArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(producer_kernel, dim3(grid), dim3(kProducerThreads), 0, s, a);
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
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, producer_kernel, kProducerThreads, 0) != hipSuccess)
    return 1;
  return n > 0 ? n : 1;
}

}  // namespace moe
