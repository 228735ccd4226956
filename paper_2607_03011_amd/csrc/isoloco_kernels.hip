// HIP kernels of the IsoLoCo outer step for gfx950 (MI355X).
//
//   reduce        K-way pseudo-gradient mean (Algorithm 1's sign, averaged as in
//                 Algorithm 2), 16-byte loads, ||Delta||_F^2 partials per chunk
//                 for the 2-D tensors (written in the iterate's column-major
//                 layout), and the whole Nesterov step (Algorithm 2) for
//                 tensors that are not corrected.
//   fro           per-matrix Frobenius norm from the partials (pre-scaling).
//   gemm          batched, grouped MFMA products (split-bf16 or fp32) for the polar iteration:
//                 Gram A = X^T X, polynomial P' = g (a I + b g^2 A + c g^4 A^2),
//                 update X <- X P'.
//   gram_norm     ||A||_F (first step: normalisation) or ||A - I||_F (check).
//   trace/sigma   sigma_bar = <Q, Delta>_F / r (mean singular value, Algorithm 2).
//   finish        fused Nesterov update and write-back of theta and B for the
//                 corrected tensors (Algorithm 2).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <mutex>

#include "isoloco.h"
#include "isoloco_kernels.h"

namespace isoloco {

// ---------------------------------------------------------------------------
// Static workspace
// ---------------------------------------------------------------------------
//
// The workspace of isoloco_aggregate_static: a fixed array in the device
// memory of every device the library runs on, held until the process ends.
// In host code the name `scratch` is a stand-in, not a device address: the
// address comes from hipGetSymbolAddress, once per device with that device
// current, and only that address is ever handed to a kernel or a copy.
static __device__ __align__(256) unsigned char scratch[ISOLOCO_STATIC_WORKSPACE_BYTES];

hipError_t static_workspace(int device, void** out) {
  constexpr int kDevices = 64;
  static std::mutex mu;
  static void* addr[kDevices] = {};
  if (device < 0 || device >= kDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[device] = p;
  }
  *out = addr[device];
  return hipSuccess;
}

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum of one value per thread over a 256-thread block, in a fixed order.
// Result valid in thread 0.
__device__ __forceinline__ double block_sum256(double v, double* lds4) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) lds4[wave] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = ((lds4[0] + lds4[1]) + lds4[2]) + lds4[3];
  return r;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// Word 3 of a raw buffer resource on CDNA3/CDNA4 (32-bit data format, no
// swizzle; the range check compares byte offsets with the record count).
constexpr int kBufferFlags = 0x00020000;
// Cache policy of the buffer loads of data read once (the "nt" bit).
constexpr int kStreamed = 2;

// A buffer resource over `bytes` bytes from p: loads at byte offsets at or
// past `bytes` return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stream_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufferFlags);
}

// ---------------------------------------------------------------------------
// K-way reduction
// ---------------------------------------------------------------------------

template <int WDT>  // 0: float32 workers, 1: bfloat16 workers
struct WorkerLoad;

template <>
struct WorkerLoad<0> {
  static constexpr int kVec = 4;  // elements per 16-byte access
  static constexpr int kBytes = 4;
  // 16 bytes at byte offset voff + soff of a stream
  __device__ static __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kStreamed));
  }
  // the 16 bytes of elements i .. i + kVec - 1, undecoded
  __device__ static __forceinline__ u32x4 raw(const void* p, int64_t i) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(static_cast<const float*>(p) + i));
  }
  __device__ static __forceinline__ float decode(const u32x4& v, int r) { return __uint_as_float(v[r]); }
  __device__ static __forceinline__ void vec(const void* p, int64_t i, float* out) {
    // replicas are read once: non-temporal loads keep them from displacing cached data
    const floatx4 v = __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(static_cast<const float*>(p) + i));
    out[0] = v[0]; out[1] = v[1]; out[2] = v[2]; out[3] = v[3];
  }
  __device__ static __forceinline__ float one(const void* p, int64_t i) {
    return static_cast<const float*>(p)[i];
  }
  __device__ static __forceinline__ void quad(const void* p, int64_t i, float* out) { vec(p, i, out); }
  // four elements, undecoded (16 bytes)
  typedef u32x4 Quad;
  __device__ static __forceinline__ Quad load_quad(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return load16(r, voff, soff);
  }
  __device__ static __forceinline__ Quad raw_quad(const void* p, int64_t i) { return raw(p, i); }
  __device__ static __forceinline__ float decode_quad(const Quad& v, int r) { return __uint_as_float(v[r]); }
};

template <>
struct WorkerLoad<1> {
  static constexpr int kVec = 8;
  static constexpr int kBytes = 2;
  __device__ static __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kStreamed));
  }
  __device__ static __forceinline__ u32x4 raw(const void* p, int64_t i) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p) + i));
  }
  // element r of the 8 bfloat16 values in v
  __device__ static __forceinline__ float decode(const u32x4& v, int r) {
    return (r & 1) ? __uint_as_float(v[r >> 1] & 0xffff0000u) : __uint_as_float(v[r >> 1] << 16);
  }
  __device__ static __forceinline__ void vec(const void* p, int64_t i, float* out) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(p) + i));
    const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(w[q] << 16);
      out[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  }
  __device__ static __forceinline__ float one(const void* p, int64_t i) {
    return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
  }
  // four elements, undecoded (8 bytes)
  typedef u32x2 Quad;
  __device__ static __forceinline__ Quad load_quad(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, kStreamed));
  }
  __device__ static __forceinline__ Quad raw_quad(const void* p, int64_t i) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(static_cast<const uint16_t*>(p) + i));
  }
  __device__ static __forceinline__ float decode_quad(const Quad& v, int r) {
    return (r & 1) ? __uint_as_float(v[r >> 1] & 0xffff0000u) : __uint_as_float(v[r >> 1] << 16);
  }
  // four elements (8 bytes)
  __device__ static __forceinline__ void quad(const void* p, int64_t i, float* out) {
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(static_cast<const uint16_t*>(p) + i));
    out[0] = __uint_as_float(v[0] << 16);
    out[1] = __uint_as_float(v[0] & 0xffff0000u);
    out[2] = __uint_as_float(v[1] << 16);
    out[3] = __uint_as_float(v[1] & 0xffff0000u);
  }
};

// Workspace index of element i of a chunk (tiles: column by column).
__device__ __forceinline__ int64_t chunk_ws(const Chunk& c, int i) {
  return c.rows ? c.ws + (int64_t)(i / c.rows) * c.ws_ld + i % c.rows : c.ws + i;
}

// LDS staging of one tile between the stored (row-major) and the workspace
// (column-major) layouts; the padded row keeps the column reads spread over
// the banks.
typedef float TileLds[kTileRows][kTileCols + 1];

// The replicas are streamed once, and the writes are what costs: the same
// loads with a store per 16-byte group run at 5.5 TB/s, the whole chunk held
// in registers and written at its end at 5.9 TB/s (probe on the 109.5M
// workload's bytes; reads alone reach 7.0 TB/s).  So every thread holds
// kSlots groups of its workgroup's chunk, walks the workers in groups whose
// loads are all in flight together (16 loads of 16 bytes per thread), and
// stores after the last worker, with non-temporal stores for Delta (read
// back only by the next kernels, from HBM).  Each element still sums
// theta - theta_k in worker order.
template <int WDT>
struct ReduceShape {
  static constexpr int kVec = WorkerLoad<WDT>::kVec;                    // elements per 16-byte load
  static constexpr int kSlots = kChunk / (kStreamThreads * kVec);       // 4 (fp32) or 2 (bf16)
  static constexpr int kGroup = 16 / kSlots;                            // workers per group
};

// Delta of a tile of a tall row-major tensor, written column-major: each
// thread reduces 8 groups of 4 consecutive stored elements of a row (a wave
// covers one row of 256 columns per group), the tile goes through LDS, and
// each thread writes 4 consecutive rows of a column (eight threads per
// 128-byte column segment).  Returns the thread's share of sum Delta^2.
// FULL: a whole kTileRows x kTileCols tile (no load needs a predicate).
template <int WDT, bool FULL>
__device__ __forceinline__ double reduce_tile(const Chunk& c, const float* __restrict__ theta,
                                              float* __restrict__ mom, float* __restrict__ delta,
                                              const WorkerPtrs& w, int K, float inv_k, float mu, int heavy_ball,
                                              int target_update, TileLds& tl) {
  using WL = WorkerLoad<WDT>;
  constexpr int S = kTileRows * (kTileCols / 4) / kStreamThreads;  // groups of 4 per thread
  constexpr int G = (WDT == 0 ? 16 : 32) / S;  // workers in flight: 256 bytes of loads per thread
  const int TR = c.rows, TC = c.cols;
  double sq = 0.0;
  if (c.vec) {
    // thread t: quad column 4 (t % 32) of rows t / 32 + 8 q (one 32-bit lane
    // offset for every slot and stream; the slot's row step is a scalar
    // offset); loads past the tile's span return zero, so none needs a
    // predicate (quads right of a narrower tile read the tensor's next row
    // and are not used)
    constexpr int kRowsPerSlot = kStreamThreads / (kTileCols / 4);
    const int r0 = threadIdx.x / (kTileCols / 4), col = 4 * (threadIdx.x % (kTileCols / 4));
    const uint32_t span = (uint32_t)((TR - 1) * c.src_ld + TC);
    const uint32_t lane = (uint32_t)(r0 * c.src_ld + col);
    const uint32_t step = (uint32_t)(kRowsPerSlot * c.src_ld);
    bool on[S];
    float th[S][4], acc[S][4];
    const __amdgpu_buffer_rsrc_t rt = stream_rsrc(theta + c.src, 4 * span);
#pragma unroll
    for (int q = 0; q < S; ++q) {
      on[q] = FULL || (r0 + kRowsPerSlot * q < TR && col < TC);
      const floatx4 t4 = __builtin_bit_cast(floatx4, WorkerLoad<0>::load16(rt, 4 * lane, 4 * step * q));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        th[q][r] = t4[r];
        acc[q][r] = 0.f;
      }
    }
#pragma unroll 1
    for (int k0 = 0; k0 < K; k0 += G) {
      // (a last group past K loads worker K - 1 again and does not add it)
      __amdgpu_buffer_rsrc_t rw[G];
#pragma unroll
      for (int j = 0; j < G; ++j)
        rw[j] = stream_rsrc(static_cast<const char*>(w.p[min(k0 + j, K - 1)]) + WL::kBytes * c.src,
                            WL::kBytes * span);
      typename WL::Quad wv[G][S];
#pragma unroll
      for (int j = 0; j < G; ++j)
#pragma unroll
        for (int q = 0; q < S; ++q) wv[j][q] = WL::load_quad(rw[j], WL::kBytes * lane, WL::kBytes * step * q);
#pragma unroll
      for (int j = 0; j < G; ++j)
        if (k0 + j < K) {
#pragma unroll
          for (int q = 0; q < S; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[q][r] += th[q][r] - WL::decode_quad(wv[j][q], r);
        }
    }
#pragma unroll
    for (int q = 0; q < S; ++q) {
      if (!on[q]) continue;
      const int rr = r0 + kRowsPerSlot * q;
      const int64_t e = c.src + (int64_t)rr * c.src_ld + col;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float a = acc[q][r] * inv_k;
        if (target_update) {
          // B <- mu B + Delta now; the polar input is the update itself
          const float bn = mu * mom[e + r] + a;
          mom[e + r] = bn;
          a = heavy_ball ? bn : a + mu * bn;
        }
        tl[rr][col + r] = a;
        sq += (double)a * a;
      }
    }
  } else {
    for (int it = threadIdx.x; it < TR * (kTileCols / 4); it += kStreamThreads) {
      const int rr = it / (kTileCols / 4), col = 4 * (it % (kTileCols / 4));
      if (col >= TC) continue;
      const int64_t e = c.src + (int64_t)rr * c.src_ld + col;
      const int nq = min(4, TC - col);
      for (int q = 0; q < nq; ++q) {
        const float th = theta[e + q];
        float acc = 0.f;
        for (int k = 0; k < K; ++k) acc += th - WL::one(w.p[k], e + q);
        float a = acc * inv_k;
        if (target_update) {
          const float bn = mu * mom[e + q] + a;
          mom[e + q] = bn;
          a = heavy_ball ? bn : a + mu * bn;
        }
        tl[rr][col + q] = a;
        sq += (double)a * a;
      }
    }
  }
  __syncthreads();
  for (int it = threadIdx.x; it < TC * (kTileRows / 4); it += kStreamThreads) {
    const int cc = it / (kTileRows / 4), r = 4 * (it % (kTileRows / 4));
    if (r >= TR) continue;
    float* dst = delta + c.ws + (int64_t)cc * c.ws_ld + r;
    if (c.vec) {
      const floatx4 o = {tl[r][cc], tl[r + 1][cc], tl[r + 2][cc], tl[r + 3][cc]};
      __builtin_nontemporal_store(o, reinterpret_cast<floatx4*>(dst));
    } else {
      for (int q = 0; q < 4 && r + q < TR; ++q) dst[q] = tl[r + q][cc];
    }
  }
  return sq;
}

// The vectorised part of a contiguous chunk: Delta of elements [0, V * (count / V))
// (ISO: stored to the workspace, returns the thread's share of sum Delta^2;
// AVG: Nesterov in place).  FULL: the chunk has kChunk elements, so every
// slot is inside it and no load needs a predicate.
template <int WDT, bool FULL>
__device__ __forceinline__ double reduce_run(const Chunk& c, float* __restrict__ theta, float* __restrict__ mom,
                                             float* __restrict__ delta, const WorkerPtrs& w, int K, float inv_k,
                                             float lr, float mu, int heavy_ball, int target_update, bool iso) {
  using WL = WorkerLoad<WDT>;
  constexpr int V = WL::kVec;
  constexpr int S = ReduceShape<WDT>::kSlots;
  constexpr int G = ReduceShape<WDT>::kGroup;
  // slot q of thread t: elements V (t + 256 q) .. +V-1 of the chunk, at byte
  // offset 16 t + 4096 q of a replica (one 32-bit lane offset for every slot
  // and stream; the slot's step is a scalar offset) and twice that for
  // bfloat16 replicas in theta; loads past the chunk return zero, so none
  // needs a predicate
  const int nv = c.count / V;
  const uint32_t lane = 16u * threadIdx.x;
  constexpr uint32_t kSlotBytes = 16u * kStreamThreads;
  bool on[S];
  float th[S][V], acc[S][V];
  const __amdgpu_buffer_rsrc_t rt = stream_rsrc(theta + c.src, 4u * (uint32_t)(nv * V));
#pragma unroll
  for (int q = 0; q < S; ++q) {
    on[q] = FULL || (int)(threadIdx.x + q * kStreamThreads) < nv;
#pragma unroll
    for (int r = 0; r < V; r += 4) {
      const floatx4 t4 = __builtin_bit_cast(
          floatx4, WorkerLoad<0>::load16(rt, lane * (V / 4) + 16u * (r / 4), kSlotBytes * (V / 4) * q));
      th[q][r] = t4[0]; th[q][r + 1] = t4[1]; th[q][r + 2] = t4[2]; th[q][r + 3] = t4[3];
    }
#pragma unroll
    for (int r = 0; r < V; ++r) acc[q][r] = 0.f;
  }
  // workers in groups of G: the group's S * G 16-byte loads are all issued
  // before any of them is consumed (differences summed in worker order)
#pragma unroll 1
  for (int k0 = 0; k0 < K; k0 += G) {
    // (a last group past K loads worker K - 1 again and does not add it)
    __amdgpu_buffer_rsrc_t rw[G];
#pragma unroll
    for (int j = 0; j < G; ++j)
      rw[j] = stream_rsrc(static_cast<const char*>(w.p[min(k0 + j, K - 1)]) + WL::kBytes * c.src,
                          WL::kBytes * (uint32_t)(nv * V));
    // the loads stay undecoded until they are added (bf16: half the registers)
    u32x4 wv[G][S];
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int q = 0; q < S; ++q) wv[j][q] = WL::load16(rw[j], lane, kSlotBytes * q);
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (k0 + j < K) {
#pragma unroll
        for (int q = 0; q < S; ++q)
#pragma unroll
          for (int r = 0; r < V; ++r) acc[q][r] += th[q][r] - WL::decode(wv[j][q], r);
      }
  }
  double sq = 0.0;
#pragma unroll
  for (int q = 0; q < S; ++q) {
    if (!on[q]) continue;
    const int v = threadIdx.x + q * kStreamThreads;
    const int64_t e = c.src + (int64_t)v * V;
#pragma unroll
    for (int r = 0; r < V; ++r) acc[q][r] *= inv_k;
    if (iso) {
      float* dst = delta + c.ws + (int64_t)v * V;
      if (target_update) {
        // B <- mu B + Delta now; the polar input is the update itself
#pragma unroll
        for (int r0 = 0; r0 < V; r0 += 4) {
          floatx4 b4 = *reinterpret_cast<const floatx4*>(mom + e + r0);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float bn = mu * b4[r] + acc[q][r0 + r];
            b4[r] = bn;
            acc[q][r0 + r] = heavy_ball ? bn : acc[q][r0 + r] + mu * bn;
          }
          *reinterpret_cast<floatx4*>(mom + e + r0) = b4;
        }
      }
#pragma unroll
      for (int r0 = 0; r0 < V; r0 += 4) {
        const floatx4 o = {acc[q][r0], acc[q][r0 + 1], acc[q][r0 + 2], acc[q][r0 + 3]};
        __builtin_nontemporal_store(o, reinterpret_cast<floatx4*>(dst + r0));
        sq += (double)o[0] * o[0] + (double)o[1] * o[1] + (double)o[2] * o[2] + (double)o[3] * o[3];
      }
    } else {
#pragma unroll
      for (int r0 = 0; r0 < V; r0 += 4) {
        floatx4 b4 = *reinterpret_cast<const floatx4*>(mom + e + r0);
        floatx4 t4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = acc[q][r0 + r];
          const float bn = mu * b4[r] + d;
          b4[r] = bn;
          t4[r] = th[q][r0 + r] - lr * (heavy_ball ? bn : d + mu * bn);
        }
        *reinterpret_cast<floatx4*>(mom + e + r0) = b4;
        *reinterpret_cast<floatx4*>(theta + e + r0) = t4;
      }
    }
  }
  return sq;
}

// Per element: Delta = (1/K) sum_k (theta - theta_k).  2-D (ISO) chunks store
// Delta in the workspace and add Delta^2 to the chunk's partial; AVG chunks run
// Nesterov in place: B <- mu B + Delta; theta <- theta - lr (Delta + mu B).
template <int WDT>
__global__ void __launch_bounds__(kStreamThreads)
reduce_kernel(const Chunk* __restrict__ chunks, float* __restrict__ theta,
              float* __restrict__ mom, float* __restrict__ delta, double* __restrict__ part_sq,
              WorkerPtrs w, int K, float inv_k, float lr, float mu, int heavy_ball, int target_update) {
  using WL = WorkerLoad<WDT>;
  constexpr int V = WL::kVec;
  __shared__ double red[4];
  __shared__ TileLds tl;
  const Chunk c = chunks[blockIdx.x];
  const bool iso = c.mat >= 0;
  double sq = 0.0;
  int done = 0;
  if (c.rows) {
    // a tile of a tall row-major tensor (always corrected): Delta column-major
    if (c.rows == kTileRows && c.cols == kTileCols)
      sq = reduce_tile<WDT, true>(c, theta, mom, delta, w, K, inv_k, mu, heavy_ball, target_update, tl);
    else
      sq = reduce_tile<WDT, false>(c, theta, mom, delta, w, K, inv_k, mu, heavy_ball, target_update, tl);
    done = c.count;
  } else if (c.vec) {
    // a whole chunk takes the path without per-slot predicates (its loads
    // are then issued back to back); a shorter last chunk of a tensor the
    // predicated one
    if (c.count == kChunk)
      sq = reduce_run<WDT, true>(c, theta, mom, delta, w, K, inv_k, lr, mu, heavy_ball, target_update, iso);
    else
      sq = reduce_run<WDT, false>(c, theta, mom, delta, w, K, inv_k, lr, mu, heavy_ball, target_update, iso);
    const int nv = c.count / V;
    done = nv * V;
  }
  for (int i = done + threadIdx.x; i < c.count; i += kStreamThreads) {
    const int64_t e = c.src + i;
    const float th = theta[e];
    float acc = 0.f;
    for (int k = 0; k < K; ++k) acc += th - WL::one(w.p[k], e);
    acc *= inv_k;
    if (iso) {
      if (target_update) {
        const float bn = mu * mom[e] + acc;
        mom[e] = bn;
        acc = heavy_ball ? bn : acc + mu * bn;
      }
      delta[c.ws + i] = acc;
      sq += (double)acc * acc;
    } else {
      const float bn = mu * mom[e] + acc;
      mom[e] = bn;
      theta[e] = th - lr * (heavy_ball ? bn : acc + mu * bn);
    }
  }
  if (iso) {
    const double s = block_sum256(sq, red);
    if (threadIdx.x == 0) part_sq[blockIdx.x] = s;
  }
}

// Sum of a matrix's chunk partials by a 256-thread block: thread t adds
// partials t, t + 256, ... in order, then block_sum256 (deterministic).
// Result valid in thread 0.
__device__ __forceinline__ double block_sum_range(const double* part, int begin, int end, double* lds4) {
  double s = 0.0;
  for (int c = begin + (int)threadIdx.x; c < end; c += 256) s += part[c];
  return block_sum256(s, lds4);
}

// Partials that one launch's workgroups hand to the last of them to arrive.
// They are stored and loaded with agent-scope atomics, which the hardware
// keeps coherent across the XCDs' separate L2 caches by themselves (no
// writeback or invalidation of a whole L2, which agent-scope release and
// acquire fences cost on this part).  arrive() waits for the workgroup's own
// store to complete before it counts itself, so that the workgroup that
// counts last finds every partial in place; it is called by one thread.
__device__ __forceinline__ void partial_store(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double partial_load(const double* p) {
  return __hip_atomic_load(const_cast<double*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Cache policy of buffer accesses at agent scope (the "sc1" bit): coherent
// across the XCDs like the atomics above.
constexpr int kAgentCoherent = 16;

// true in the workgroup that is the n-th to arrive at *cnt, which it sets back to zero
__device__ __forceinline__ bool arrive(int* cnt, int n) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  const bool last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n - 1;
  asm volatile("" ::: "memory");
  if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return last;
}

// ||Delta||_F per matrix (one block per matrix).
__global__ void __launch_bounds__(256)
fro_kernel(const MatInfo* __restrict__ mats, const double* __restrict__ part_sq,
           MatScalars* __restrict__ sc, int n_mat, FroArgs a) {
  __shared__ double red[4];
  const int m = blockIdx.x;
  const MatInfo mi = mats[m];
  const double s = block_sum_range(part_sq, mi.chunk_begin, mi.chunk_end, red);
  if (threadIdx.x != 0) return;
  MatScalars o;
  o.fro = (float)sqrt(s);
  o.flags = 0;
  if (!isfinite(s)) o.flags |= kFlagNonfinite;
  else if (s == 0.0) o.flags |= kFlagZero;
  o.inv_fro = (o.flags == 0) ? (float)(1.0 / sqrt(s)) : 0.f;
  o.gscale = (a.fixed_g && o.flags == 0) ? 1.f : 0.f;  // else set from the first Gram
  o.sigma_bar = 0.f;
  o.resid = -1.f;
  o.steps = a.steps_total[mi.sched];
  o.active = 1;
  o.qbuf = a.buf_total[mi.sched];
  sc[m] = o;
}

// ---------------------------------------------------------------------------
// Batched fp32 MFMA products of the polar iteration
// ---------------------------------------------------------------------------
//
// Output tile 128 x 128 per 256-thread workgroup; wave w owns the 64 x 64
// quarter (w >> 1, w & 1) as 2 x 2 blocks of v_mfma_f32_32x32x2f32.  K is
// staged through LDS in slabs of 16, with the next slab's global loads in
// flight while the current one is multiplied.  LDS holds both operands
// k-major ([k][i], i contiguous) so that a wavefront's operand read is two
// rows of 32 consecutive floats.

constexpr int kLdsW = kBM + 4;

// A 16 x 128 operand slab: element (k, i) at base + k * s_k + i * s_i, with
// either s_i == 1 ("i-contiguous") or s_k == 1 ("k-contiguous").
struct Operand {
  const float* base;
  int64_t s_k, s_i;
  int K, I;       // bounds: k in [0, K), i in [0, I)
  bool icontig;
  bool vec;
  float scale;
};

struct SlabRegs {
  floatx4 v[2];
};

__device__ __forceinline__ void slab_load(const Operand& op, int k0, int i0, SlabRegs& r) {
  const int t = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    floatx4 x = {0.f, 0.f, 0.f, 0.f};
    if (op.icontig) {
      const int k = k0 + (t >> 5) + 8 * rep;
      const int i = i0 + 4 * (t & 31);
      if (k < op.K) {
        const float* p = op.base + (int64_t)k * op.s_k + i;
        if (op.vec && i + 3 < op.I) {
          x = *reinterpret_cast<const floatx4*>(p);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (i + e < op.I) x[e] = p[e];
        }
      }
    } else {
      const int i = i0 + (t >> 2) + 64 * rep;
      const int k = k0 + 4 * (t & 3);
      if (i < op.I) {
        const float* p = op.base + (int64_t)i * op.s_i + k;
        if (op.vec && k + 3 < op.K) {
          x = *reinterpret_cast<const floatx4*>(p);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (k + e < op.K) x[e] = p[e];
        }
      }
    }
    r.v[rep] = x * op.scale;
  }
}

__device__ __forceinline__ void slab_store(const Operand& op, const SlabRegs& r, float (*lds)[kLdsW]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    if (op.icontig) {
      const int k = (t >> 5) + 8 * rep;
      const int i = 4 * (t & 31);
      *reinterpret_cast<floatx4*>(&lds[k][i]) = r.v[rep];
    } else {
      const int i = (t >> 2) + 64 * rep;
      const int k = 4 * (t & 3);
#pragma unroll
      for (int e = 0; e < 4; ++e) lds[k + e][i] = r.v[rep][e];
    }
  }
}

enum GemmMode { kGram = 0, kPoly = 1, kUpdate = 2 };

struct GemmArgs {
  const MatInfo* mats;
  const Task* tasks;
  const MatScalars* sc;
  MatScalars* sc_out;  // Gram with norm_mode >= 0: the same scalars, which the decisions write
  const float* xin;   // Gram/Update: X input buffer (Delta at step 0)
  const float* xin_alt;  // Gram: if set, matrices whose qbuf is 1 read X here
  const float* bin;      // Gram: if set, the second operand B (C = X^T B)
  float* xout;        // Update: X output buffer
  float* gram;        // n x n Gram buffers (Gram output, Poly input)
  float* poly;        // n x n polynomial buffers (Poly output, Update input)
  float* gpart;       // split-K Gram partials
  int* split_cnt;     // split-K Gram: arrival counter per output tile
  int* mat_cnt;       // Gram with norm_mode >= 0: arrival counter per matrix
  double* part_norm;  // Gram: per-tile partial sums of squares (norm_mode >= 0)
  const float* coef;  // Poly: coefficients [class][n_steps][3] of p(x) = ca x + cb x^3 + cc x^5
  int step, n_steps;  // Poly: this step, and the table's steps per class
  int first;          // 1 on the first step (inputs pre-scaled by 1/||Delta||_F, g applied)
  int only_active;    // 1: tasks of matrices that stopped iterating return at once
  int norm_mode;      // Gram: -1, or kNormFirst (sum A^2) / other (sum (A - I)^2) per tile
  NormArgs na;        // norm_mode >= 0: the decisions of the matrix's last tile (norm_decide)
};

// Operands, output bounds and K range of one task.
//   Gram:    C(i, j) = sum_k X[k][i] X[k][j]   over the task's K slice (C is n x n)
//   Poly:    C(i, j) = sum_k A[i][k] A[j][k]   (A symmetric, so this is A A)
//   Update:  C(i, j) = sum_k X[i][k] P[k][j]   (C is m x n, tall coordinates)
struct GemmSetup {
  MatInfo mi;
  Operand A, B;
  int M, N, k_begin, k_end, i0, j0;
  int64_t sr, sc;
  float xscale;  // applied to X operands as they are loaded (1/||Delta||_F on the first step)
  float gs;      // normalisation g of the first step (1 afterwards)
  float ca, cb, cc;  // Poly: this matrix's step coefficients (its schedule class)
};

template <int MODE, int TILE = kBM>
__device__ __forceinline__ GemmSetup gemm_setup(const GemmArgs& g, const Task& task) {
  GemmSetup s;
  s.mi = g.mats[task.mat];
  const MatInfo& mi = s.mi;
  const int m = mi.m, n = mi.n;
  // every iterate is column-major in tall coordinates: X[r][c] at r + c m
  s.sr = 1;
  s.sc = m;
  const bool vec = mi.vec != 0;
  s.xscale = 1.f;
  s.gs = 1.f;
  if (g.first) {
    const MatScalars q = g.sc[task.mat];
    s.xscale = q.inv_fro;
    s.gs = q.gscale;
  }
  if (MODE == kGram) {
    const float* x = ((g.xin_alt && g.sc[task.mat].qbuf) ? g.xin_alt : g.xin) + mi.ws_off;
    s.k_begin = task.ks * mi.kchunk;
    s.k_end = min(m, s.k_begin + mi.kchunk);
    s.A = {x, s.sr, s.sc, s.k_end, n, false, vec, s.xscale};
    s.B = s.A;
    if (g.bin) s.B.base = g.bin + mi.ws_off;
    s.M = n;
    s.N = n;
  } else if (MODE == kPoly) {
    const float* c = g.coef + ((int64_t)mi.sched * g.n_steps + g.step) * 3;
    s.ca = c[0];
    s.cb = c[1];
    s.cc = c[2];
    const float* a = g.gram + mi.sq_off;
    // A is symmetric (its diagonal tiles to rounding), so the operand A[k][i]
    // is read as A[i][k]: k-contiguous rows, the faster loads
    s.A = {a, 1, (int64_t)n, n, n, false, (n & 3) == 0, 1.f};
    s.B = s.A;
    s.M = n;
    s.N = n;
    s.k_begin = 0;
    s.k_end = n;
  } else {
    const float* x = g.xin + mi.ws_off;
    s.A = {x, s.sc, s.sr, n, m, true, vec, s.xscale};
    const float* p = g.poly + mi.sq_off;
    s.B = {p, (int64_t)n, 1, n, n, true, (n & 3) == 0, 1.f};
    s.M = m;
    s.N = n;
    s.k_begin = 0;
    s.k_end = n;
  }
  s.i0 = task.tm * TILE;
  s.j0 = task.tn * TILE;
  return s;
}

// Accumulator start values.  Zero, except for the polynomial product, whose
// epilogue forms P' = g (a I + b g^2 A + c g^4 A^2) = gamma (rho A + A A) +
// a g I with gamma = c g^5 and rho = b / (c g^2): the accumulators start at
// rho A(i, j), read here with the first operand slabs in flight, so that the
// epilogue does not wait on a second read of A.  (The schedule's quintics all
// have c != 0.)  A is symmetric: A(i, j) is read as the 4 consecutive
// values A(j, i .. i + 3) that one lane holds in the accumulator layout.
template <int MODE, int NA = 2, int WNC = 2>
__device__ __forceinline__ void gemm_acc_init(const GemmArgs& g, const GemmSetup& s, floatx16 (&acc)[NA][2]) {
  if (MODE != kPoly) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
    return;
  }
  const int n = s.mi.n;
  // (g = 0 marks a zero or non-finite Delta: P' = 0 then, and rho is kept finite)
  const float rho = s.gs != 0.f ? s.cb / (s.cc * s.gs * s.gs) : 0.f;
  const float* A = g.gram + s.mi.sq_off;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WNC, wn = wave % WNC;
  const bool v4 = (n & 3) == 0;
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int j = s.j0 + wn * 64 + b * 32 + (lane & 31);
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int ib = s.i0 + wm * 32 * NA + a * 32 + 8 * grp + 4 * (lane >> 5);
        floatx4 v = {0.f, 0.f, 0.f, 0.f};
        if (j < n) {
          const float* row = A + (int64_t)j * n + ib;
          if (v4 && ib + 3 < n) {
            v = *reinterpret_cast<const floatx4*>(row);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (ib + r < n) v[r] = row[r];
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[a][b][4 * grp + r] = rho * v[r];
      }
    }
}

// The decisions of matrix mi from its Gram's norm partials (see NormMode,
// NormAction): the partials of its gram_tiles(n) tiles are added in tile order.
__device__ __forceinline__ void norm_decide(const MatInfo& mi, const double* part, MatScalars& o, const NormArgs& a) {
  if (a.cls >= 0 && mi.sched != a.cls) return;
  const int act = a.mode == kNormFirst ? kActNone : a.action[mi.sched];
  if (a.mode != kNormFirst && act == kActNone) return;
  if (act == kActStop) {
    o.active = 0;
    return;
  }
  double s = 0.0;
  const int nt = gram_tiles(mi.n);
  for (int x = 0; x < nt; ++x) s += partial_load(part + mi.norm_off + x);
  if (a.mode == kNormFirst) {
    o.gscale = ((o.flags & kFlagInput) == 0 && s > 0.0) ? (float)(1.0 / sqrt(sqrt(s))) : 0.f;
    return;
  }
  o.resid = (float)sqrt(s / mi.n);
  if (act == kActSwitch) {
    // stop at the end of this phase when every singular value is already at 1
    const bool go_on = (o.flags & kFlagInput) == 0 && !(o.resid <= a.tol_switch);
    // a matrix that still has a singular value away from 1 after the schedule
    // for a bound at the float32 resolution of Delta has one below it: its
    // direction in Q is decided by rounding, not by Delta
    if (go_on && a.flag_below[mi.sched]) o.flags |= kFlagBelowResolution;
    o.active = go_on ? 1 : 0;
    o.steps = go_on ? a.steps_total[mi.sched] : a.steps_here;
    o.qbuf = go_on ? a.buf_total[mi.sched] : a.buf_here;
  } else {
    if (a.flag_unconverged && !(o.resid <= 1e-3f) && (o.flags & kFlagInput) == 0) o.flags |= kFlagNotConverged;
    o.active = 0;
  }
}

// Gram epilogue.  Writes the tile and its mirror image into the n x n Gram
// buffer and, when the launch asks for it, the tile's share of ||A||_F^2 or
// ||A - I||_F^2 (twice the tile's sum off the diagonal) into its slot of
// part_norm.  The last tile of a matrix to arrive (counted per matrix like the
// split-K slices below) adds the matrix's slots in a fixed order and takes its
// decisions (norm_decide), so that no launch of its own is needed for them.
//
// A split-K matrix first writes this K slice's partial tile into its slice of
// gpart.  The last of the ksplit workgroups of a tile to arrive (arrive(),
// with the partials stored and loaded at agent scope so that those written on
// other XCDs are seen) adds the slices in slice order and finishes the tile as
// above.  No workgroup waits for another.  `scratch` is LDS the operand
// planes no longer need (at least 40 bytes).
template <int NA, int WNC>
__device__ __forceinline__ void gram_epilogue(const GemmArgs& g, const GemmSetup& s, const Task& task,
                                              const floatx16 (&acc)[NA][2], void* scratch) {
  const MatInfo& mi = s.mi;
  const int n = mi.n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WNC, wn = wave % WNC;
  const int jl = lane & 31, ib = 4 * (lane >> 5);
  const int tile = gram_tile_index(n, task.tm, task.tn);
  double* red = reinterpret_cast<double*>(scratch);
  int* last = reinterpret_cast<int*>(red + 4);
  floatx16 v[NA][2];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) v[a][b] = acc[a][b];
  if (mi.ksplit > 1) {
    // partial tiles are stored transposed (C(i, j) at j * n + i), so that the
    // 4 values a lane holds, C(i .. i+3, j), are one 16-byte access; they are
    // stored and loaded at agent scope (the planner keeps a matrix's slices
    // under 2 GiB, the range of the buffer offsets)
    const int64_t nn = (int64_t)n * n;
    const bool v4 = (n & 3) == 0;
    const __amdgpu_buffer_rsrc_t pr = stream_rsrc(g.gpart + mi.part_off, (uint32_t)(4 * mi.ksplit * nn));
    const int64_t mine = (int64_t)task.ks * nn;
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int j = s.j0 + wn * 64 + b * 32 + jl;
        if (j >= s.N) continue;
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int ibase = s.i0 + wm * 32 * NA + a * 32 + 8 * grp + ib;
          const int off = (int)(4 * (mine + (int64_t)j * n + ibase));
          if (v4 && ibase + 3 < s.M) {
            const floatx4 q = {v[a][b][4 * grp], v[a][b][4 * grp + 1], v[a][b][4 * grp + 2], v[a][b][4 * grp + 3]};
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, q), pr, off, 0, kAgentCoherent);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (ibase + r < s.M)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[a][b][4 * grp + r]), pr, off + 4 * r, 0,
                                                      kAgentCoherent);
          }
        }
      }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's slice is in place
    __syncthreads();  // every wave's partial is out, and the operand planes are free
    if (threadIdx.x == 0) *last = arrive(g.split_cnt + mi.cnt_off + tile, mi.ksplit);
    __syncthreads();
    if (!*last) return;
    // the slices in slice order; every load of the tile is independent of the
    // sums, so that they can all be in flight together
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int j = s.j0 + wn * 64 + b * 32 + jl;
        if (j >= s.N) continue;
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int ibase = s.i0 + wm * 32 * NA + a * 32 + 8 * grp + ib;
          const bool vec = v4 && ibase + 3 < s.M;
          const floatx4 own = {v[a][b][4 * grp], v[a][b][4 * grp + 1], v[a][b][4 * grp + 2], v[a][b][4 * grp + 3]};
          floatx4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int k = 0; k < kMaxKSplit; ++k) {
            if (k >= mi.ksplit) break;
            floatx4 x = own;
            if (k != task.ks) {
              const int off = (int)(4 * (k * nn + (int64_t)j * n + ibase));
              if (vec) {
                x = __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(pr, off, 0, kAgentCoherent));
              } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  x[r] = ibase + r < s.M
                             ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(pr, off + 4 * r, 0, kAgentCoherent))
                             : 0.f;
              }
            }
            t = k == 0 ? x : t + x;
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) v[a][b][4 * grp + r] = t[r];
        }
      }
  }
  float* out = g.gram + mi.sq_off;
  const bool diag = task.tm == task.tn;
  const bool want = g.norm_mode >= 0;
  const float unit = g.norm_mode == kNormFirst ? 0.f : 1.f;
  double sq = 0.0;
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int j = s.j0 + wn * 64 + b * 32 + jl;
      if (j >= s.N) continue;
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int ibase = s.i0 + wm * 32 * NA + a * 32 + 8 * grp + ib;
        floatx4 q;
#pragma unroll
        for (int r = 0; r < 4; ++r) q[r] = v[a][b][4 * grp + r];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = ibase + r;
          if (i >= s.M) continue;
          out[(int64_t)i * n + j] = q[r];
          if (want) {
            const double d = (double)q[r] - (i == j ? unit : 0.f);
            sq += d * d;
          }
        }
        if (!diag) {
          float* mo = out + (int64_t)j * n + ibase;
          if ((n & 3) == 0 && ibase + 3 < s.M) {
            *reinterpret_cast<floatx4*>(mo) = q;
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (ibase + r < s.M) mo[r] = q[r];
          }
        }
      }
    }
  if (want) {
    __syncthreads();  // the operand planes are free (split tiles passed this point already)
    sq = block_sum256(sq, red);
    if (threadIdx.x == 0) {
      partial_store(g.part_norm + mi.norm_off + tile, diag ? sq : 2.0 * sq);
      if (arrive(g.mat_cnt + task.mat, gram_tiles(n))) norm_decide(mi, g.part_norm, g.sc_out[task.mat], g.na);
    }
  }
}

// Epilogue.  A wave owns NA x 2 accumulator tiles of 32 x 32: with WNC waves
// across the block's columns, wm = wave / WNC and wn = wave % WNC,
// acc[a][b][r] holds C(i, j) with
//   i = i0 + wm*32*NA + a*32 + 8*(r/4) + 4*(lane/32) + r%4,  j = j0 + wn*64 + b*32 + lane%32
// (the 32 x 32 accumulator layout of the fp32 and bf16 MFMA instructions).
// Interior update tiles of the split-bf16 kernels store through
// store_update_colmajor instead.
template <int MODE, int NA = 2, int WNC = 2>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, const GemmSetup& s, const Task& task,
                                              const floatx16 (&acc)[NA][2], void* scratch = nullptr) {
  if constexpr (MODE == kGram) {
    gram_epilogue<NA, WNC>(g, s, task, acc, scratch);
    return;
  }
  const MatInfo& mi = s.mi;
  const int n = mi.n;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WNC, wn = wave % WNC;
  const int jl = lane & 31;
  const int ib = 4 * (lane >> 5);
#pragma unroll
  for (int a = 0; a < NA; ++a) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int j = s.j0 + wn * 64 + b * 32 + jl;
      if (j >= s.N) continue;
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int ibase = s.i0 + wm * 32 * NA + a * 32 + 8 * grp + ib;
        if (MODE == kPoly) {
          // symmetric n x n result: only tiles with tm <= tn are computed, and an
          // off-diagonal tile also writes its mirror image C(j, i) = C(i, j).
          // P = g (ca I + cb g^2 A + cc g^4 A^2)  (g = 1 after the first step),
          // so that the update is the plain product X' = X P; the accumulators
          // hold rho A + A A (see gemm_acc_init)
          const float g2 = s.gs * s.gs;
          const float gamma = s.cc * g2 * g2 * s.gs, diag = s.ca * s.gs;
          float* out = g.poly + mi.sq_off;
          floatx4 v;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = ibase + r;
            v[r] = gamma * acc[a][b][4 * grp + r] + (i == j ? diag : 0.f);
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = ibase + r;
            if (i < s.M) out[(int64_t)i * n + j] = v[r];
          }
          if (task.tm != task.tn) {
            float* mo = out + (int64_t)j * n + ibase;
            if ((n & 3) == 0 && ibase + 3 < s.M) {
              *reinterpret_cast<floatx4*>(mo) = v;
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (ibase + r < s.M) mo[r] = v[r];
            }
          }
        } else {
          // X' = X P (the linear term and g are folded into P)
          float* xo = g.xout + mi.ws_off;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = ibase + r;
            if (i < s.M) xo[(int64_t)i * s.sr + (int64_t)j * s.sc] = acc[a][b][4 * grp + r];
          }
        }
      }
    }
  }
}

// fp32 MFMA main loop (v_mfma_f32_32x32x2f32), K staged in slabs of 16.
template <int MODE>
__global__ void __launch_bounds__(kGemmThreads, 2) gemm_f32_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) float As[kBK][kLdsW];
  __shared__ __attribute__((aligned(16))) float Bs[kBK][kLdsW];
  const Task task = g.tasks[blockIdx.x];
  if (task.mat < 0 || (g.only_active && !g.sc[task.mat].active)) return;
  const GemmSetup s = gemm_setup<MODE>(g, task);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  floatx16 acc[2][2];
  gemm_acc_init<MODE>(g, s, acc);

  SlabRegs ra, rb;
  slab_load(s.A, s.k_begin, s.i0, ra);
  slab_load(s.B, s.k_begin, s.j0, rb);
  for (int k0 = s.k_begin; k0 < s.k_end; k0 += kBK) {
    slab_store(s.A, ra, As);
    slab_store(s.B, rb, Bs);
    __syncthreads();
    if (k0 + kBK < s.k_end) {
      slab_load(s.A, k0 + kBK, s.i0, ra);
      slab_load(s.B, k0 + kBK, s.j0, rb);
    }
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 2) {
      const int kr = kk + (lane >> 5);
      const float a0 = As[kr][wm * 64 + (lane & 31)];
      const float a1 = As[kr][wm * 64 + 32 + (lane & 31)];
      const float b0 = Bs[kr][wn * 64 + (lane & 31)];
      const float b1 = Bs[kr][wn * 64 + 32 + (lane & 31)];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    __syncthreads();
  }
  gemm_epilogue<MODE>(g, s, task, acc, &As[0][0]);
}

// ---------------------------------------------------------------------------
// Split-bfloat16 main loop (bf16x3, bf16x5 and bf16x6)
// ---------------------------------------------------------------------------
//
// Each fp32 operand x is split into NS bfloat16 parts, x = x0 + x1 (+ x2) + r,
// x0 = bf16(x), x1 = bf16(x - x0), x2 = bf16(x - x0 - x1), round to nearest
// even, so |r| <= 2^-16 |x| for NS = 2 and 2^-24 |x| for NS = 3.  The product
// sum_k a_k b_k is accumulated in fp32 over the part products of order
// i + j <= 2 that both splits provide:
//   bf16x3 (2 + 2 parts):  a1 b0 + a0 b1 + a0 b0
//   bf16x5 (3 + 2 parts):  a2 b0 + a1 b1 + a1 b0 + a0 b1 + a0 b0
//   bf16x6 (3 + 3 parts):  a2 b0 + a1 b1 + a0 b2 + a1 b0 + a0 b1 + a0 b0
// on v_mfma_f32_32x32x16_bf16.  K is staged in slabs of 32: fp32 global loads
// into registers (next slab in flight during the current slab's products),
// split, and stored to LDS as NS bf16 planes per operand in [row][k] order, so
// that every lane reads its 8 consecutive k values of a row with one 16-byte
// LDS read.

constexpr int kBK2 = 32;
constexpr int kLdsK = kBK2 + 8;  // padded row (bf16 elements): 80 bytes

// Element offset within an LDS operand row of its 16-byte k-chunk c (0..3).
// Rows of LK = 40 bf16 (80 bytes) keep 16-byte accesses to 16 consecutive
// rows on distinct banks as they are (an LDS of 64 banks serves 16 lanes of a
// 16-byte access per pass).  Rows of LK = 32 (64 bytes, no padding: room for
// two buffers of bf16x5 operands) XOR the chunk position with bits 1-2 of the
// row XOR bits 2-3: the four rows that share a set of 16 banks (r, r + 4,
// r + 8, r + 12) then take four different chunk positions.  (Bits 1-2 alone
// spread 8 consecutive rows only, which leaves 2-way conflicts on 64 banks.)
template <int LK>
__device__ __forceinline__ int lds_chunk(int row, int c) {
  static_assert(LK == kLdsK || LK == kBK2, "80- or 64-byte operand rows");
  return LK == kBK2 ? ((c ^ (((row >> 1) ^ (row >> 2)) & 3)) << 3) : (c << 3);
}

// Row of the slab covered by thread t's group of eight lanes in the row
// mapping (each group stores one row's 64 bytes of a plane with 8-byte
// writes).  With 80-byte LDS rows, rows r and r + 1 share banks, so the
// groups take t / 8 with bits 0-1 and 2-3 swapped: the groups of one pass
// (two of 16 lanes, or four of 32) store rows r, r + 4, r + 8, r + 12, which
// fall on distinct banks.  64-byte rows keep t / 8 (their chunk swizzle
// spreads consecutive rows already).
template <int LK>
__device__ __forceinline__ int rowmap_row(int t) {
  const int g = t >> 3;
  return LK == kBK2 ? g : (g & ~15) | ((g & 3) << 2) | ((g >> 2) & 3);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct Slab32 {
  floatx4 v[4];
};


// 128 (i) x 32 (k) fp32 slab into registers: thread t owns row i = t % 128
// and the 16 consecutive k values 16 (t / 128) .. +15, so that its LDS writes
// are 16-byte row segments and consecutive lanes write consecutive rows
// (80-byte stride: no bank conflicts).  SCALED multiplies by the operand's
// scale (the 1/||Delta||_F of the first polar step; 1 afterwards, when the
// multiply is left out).
// Interior slab (no bounds checks; the host only routes tiles whose rows,
// columns and K range are all inside the matrix, with m, n multiples of 4).
// ROWS = 128 (256 threads) or 256 (512 threads): the slab is ROWS x 32 and
// every thread holds 16 of its values.
template <bool ICONTIG, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void slab32_load_fast(const Operand& op, int k0, int i0, Slab32& r) {
  const int t = threadIdx.x;
  // Buffer loads: a uniform resource for the operand's matrix, one 32-bit lane
  // offset that is fixed for the whole slab, and the k advance as a scalar
  // offset, so that no per-load address arithmetic runs on the vector ALU.
  // The host keeps matrices of these tiles under 2^29 elements, so every byte
  // offset fits 31 bits.
  const int bytes = 4 * ((op.K - 1) * (int)op.s_k + (op.I - 1) * (int)op.s_i + 1);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(op.base), (short)0, bytes, kBufferFlags);
  if (ICONTIG) {
    // element (k, i) at base + k s_k + i: thread t holds row i0 + t % ROWS and
    // k = k0 + 16 (t / ROWS) .. +15; lanes take consecutive i (coalesced 4-byte
    // loads); t / ROWS is uniform over a wave
    const int kb = k0 + 16 * __builtin_amdgcn_readfirstlane(t / ROWS);
    const int vo = 4 * (i0 + t % ROWS);
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        r.v[q][e] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(rs, vo, 4 * (kb + 4 * q + e) * (int)op.s_k, 0));
  } else {
    // element (k, i) at base + i s_i + k: row mapping -- eight lanes cover the
    // slab's 128 contiguous bytes of one row, a wave eight rows per load
    // (thread t: rows i0 + rowmap_row(t) + (ROWS / 4) q, k = k0 + 4 (t % 8)
    // .. +3), so that a load touches 8 cache lines instead of 64
    const int vo = 4 * ((i0 + rowmap_row<LK>(t)) * (int)op.s_i + 4 * (t & 7));
#pragma unroll
    for (int q = 0; q < 4; ++q)
      r.v[q] = __builtin_bit_cast(
          floatx4, __builtin_amdgcn_raw_buffer_load_b128(rs, vo, 4 * (k0 + (ROWS / 4) * q * (int)op.s_i), 0));
  }
}

// Any slab: runtime layout, every element bounds-checked (zero outside).
__device__ __forceinline__ void slab32_load(const Operand& op, int k0, int i0, Slab32& r) {
  const int t = threadIdx.x;
  const int i = i0 + (t & 127);
  const int kb = k0 + 16 * (t >> 7);
  if (op.icontig) {
    const float* p = op.base + (int64_t)kb * op.s_k + i;
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = kb + 4 * q + e;
        r.v[q][e] = (i < op.I && k < op.K) ? p[(int64_t)(4 * q + e) * op.s_k] : 0.f;
      }
  } else {
    const float* p = op.base + (int64_t)i * op.s_i + kb;
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = kb + 4 * q + e;
        r.v[q][e] = (i < op.I && k < op.K) ? p[4 * q + e] : 0.f;
      }
  }
}

// Loader selected at compile time: LAYOUT kGeneric uses runtime layout and
// bounds; the fast layouts fix the contiguity of the A and B operands.
// kFast: interior tiles, unchecked buffer loads of the operands' fixed
// layout; kGeneric: ragged tiles and matrices too large for 32-bit offsets,
// bounds-checked loads of either layout.
enum TileLayout { kGeneric = 0, kFast = 1 };

// Operands of the interior tiles (the iterates column-major): Gram, both X[k][i]
// with k contiguous; Poly, A[k][i] read as A[i][k] (symmetric), k-contiguous;
// Update, A = X[i][k] and B = P[k][j], both i-contiguous.  k-contiguous
// operands use the row mapping of the registers.
template <int MODE, int LAYOUT>
struct OperandLayout {
  static constexpr bool icontig = MODE == kUpdate;
  static constexpr bool rowmap = LAYOUT != kGeneric && !icontig;
};

template <int MODE, int LAYOUT, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void load_operand(const Operand& op, int k0, int i0, Slab32& r) {
  static_assert(LAYOUT != kGeneric || ROWS == kBM, "ragged tiles use the 128-row kernel");
  if (LAYOUT == kGeneric) slab32_load(op, k0, i0, r);
  else slab32_load_fast<OperandLayout<MODE, LAYOUT>::icontig, ROWS, LK>(op, k0, i0, r);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Split the thread's 16 values into NS bf16 parts, two values per convert,
// and store each part plane as two 16-byte row segments.  SCALED multiplies
// the values by the operand's scale first (the 1/||Delta||_F of the first
// polar step; 1 afterwards, when the multiply is left out).
template <int NS, bool SCALED = false, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void slab32_store(const Slab32& r, __bf16 (*planes)[ROWS][LK], float scale = 1.f) {
  const int t = threadIdx.x;
  const int i = t % ROWS, kb = 16 * (t / ROWS);
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    bf16x8 part[NS];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      floatx2 x = {r.v[2 * half + e / 4][e % 4], r.v[2 * half + e / 4][e % 4 + 1]};
      if (SCALED) x *= scale;
#pragma unroll
      for (int p = 0; p < NS; ++p) {
        const bf16x2 h = __builtin_convertvector(x, bf16x2);
        part[p][e] = h[0];
        part[p][e + 1] = h[1];
        if (p + 1 < NS) x -= __builtin_convertvector(h, floatx2);
      }
    }
#pragma unroll
    for (int p = 0; p < NS; ++p)
      *reinterpret_cast<bf16x8*>(&planes[p][i][lds_chunk<LK>(i, (kb >> 3) + half)]) = part[p];
  }
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// The same for registers in the row mapping (thread t: rows rowmap_row(t) +
// (ROWS / 4) q, k = 4 (t % 8) .. +3): 8-byte LDS writes.
template <int NS, bool SCALED = false, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void slab32_store_rows(const Slab32& r, __bf16 (*planes)[ROWS][LK], float scale = 1.f) {
  const int t = threadIdx.x;
  const int i = rowmap_row<LK>(t), kb = 4 * (t & 7);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bf16x4 part[NS];
#pragma unroll
    for (int e = 0; e < 4; e += 2) {
      floatx2 x = {r.v[q][e], r.v[q][e + 1]};
      if (SCALED) x *= scale;
#pragma unroll
      for (int p = 0; p < NS; ++p) {
        const bf16x2 h = __builtin_convertvector(x, bf16x2);
        part[p][e] = h[0];
        part[p][e + 1] = h[1];
        if (p + 1 < NS) x -= __builtin_convertvector(h, floatx2);
      }
    }
    const int row = i + (ROWS / 4) * q;
#pragma unroll
    for (int p = 0; p < NS; ++p)
      *reinterpret_cast<bf16x4*>(&planes[p][row][lds_chunk<LK>(row, kb >> 3) + (kb & 7)]) = part[p];
  }
}

template <int MODE, int LAYOUT, int NS, bool SCALED, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void store_operand(const Slab32& r, __bf16 (*planes)[ROWS][LK], float scale) {
  if (OperandLayout<MODE, LAYOUT>::rowmap) slab32_store_rows<NS, SCALED, ROWS, LK>(r, planes, scale);
  else slab32_store<NS, SCALED, ROWS, LK>(r, planes, scale);
}

// Split-bf16 arithmetic with NP part products per fp32 product: NP = 3
// (bf16x3: both operands in 2 parts, products of part orders 0 + 0, 0 + 1,
// 1 + 0), NP = 6 (bf16x6: 3 parts each, all orders up to 2) and NP = 5 (left
// operand in 3 parts, right operand in 2: the orders up to 2 without the
// right operand's third part).  NP = 5 serves the update X' = X P': a
// rounding error of X enters every direction of X' with the size of X's
// largest singular values, while an error of P' enters the component of
// each singular direction in proportion to its singular value, so the left
// factor needs the third part and the right factor does not.
template <int NP>
struct SplitParts {
  static_assert(NP == 3 || NP == 5 || NP == 6, "bf16x3, bf16x5 or bf16x6");
  static constexpr int a = NP == 3 ? 2 : 3;   // planes of the left operand
  static constexpr int b = NP == 6 ? 3 : 2;   // planes of the right operand
  static constexpr int nb = NP == 3 ? 2 : 1;  // LDS buffers (double-buffered bf16x3)
};

// One k16 substep of a wave's (32 NA) x 64 tile: read the operand fragments
// of the NSA / NSB planes from LDS and issue the part products (smallest
// order first).  WNC waves span the block's columns (wm = wave / WNC,
// wn = wave % WNC).
template <int NSA, int NSB, int NA = 2, int WNC = 2, int ROWS = kBM, int LK = kLdsK>
__device__ __forceinline__ void mfma_substep(const __bf16 (*Ap)[ROWS][LK], const __bf16 (*Bp)[ROWS][LK],
                                             int kk, floatx16 (&acc)[NA][2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WNC, wn = wave % WNC;
  const int kc = kk + 8 * (lane >> 5);
  constexpr int kMaxOrd = (NSA > NSB ? NSA : NSB) - 1;
  bf16x8 av[NA][NSA], bv[2][NSB];
#pragma unroll
  for (int a = 0; a < NA; ++a) {
    const int row = wm * 32 * NA + a * 32 + (lane & 31);
#pragma unroll
    for (int p = 0; p < NSA; ++p) av[a][p] = *reinterpret_cast<const bf16x8*>(&Ap[p][row][lds_chunk<LK>(row, kc >> 3)]);
  }
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int row = wn * 64 + b * 32 + (lane & 31);
#pragma unroll
    for (int p = 0; p < NSB; ++p) bv[b][p] = *reinterpret_cast<const bf16x8*>(&Bp[p][row][lds_chunk<LK>(row, kc >> 3)]);
  }
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int ord = kMaxOrd; ord >= 0; --ord)
#pragma unroll
        for (int pa = ord; pa >= 0; --pa) {
          const int pb = ord - pa;
          if (pa >= NSA || pb >= NSB) continue;
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[a][pa], bv[b][pb], acc[a][b], 0, 0, 0);
        }
}

// Interior update tile of a column-major X': the accumulators of each
// 32-column block go through the wave's own LDS region (columns padded to
// 32 NA + 4 floats), so that every store instruction writes whole columns
// of the wave's 32 NA rows -- full 128-byte lines -- instead of 32-byte
// pieces of 32 columns.
template <int NA>
__host__ __device__ constexpr int stage_floats(int waves) { return waves * 32 * (32 * NA + 4); }

template <int NA, int WNC>
__device__ __forceinline__ void store_update_colmajor(const GemmArgs& g, const GemmSetup& s,
                                                      const floatx16 (&acc)[NA][2], float* stage) {
  constexpr int RW = 32 * NA;     // rows of the wave's tile
  constexpr int LD = RW + 4;      // padded LDS column
  constexpr int LPC = RW / 4;     // lanes per column in a store
  constexpr int CPI = 64 / LPC;   // columns per store instruction
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WNC, wn = wave % WNC;
  float* ws = stage + wave * 32 * LD;
  float* xo = g.xout + s.mi.ws_off;
  __syncthreads();  // every wave is done with the operand planes
#pragma unroll
  for (int b = 0; b < 2; ++b) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const floatx4 v = {acc[a][b][4 * grp], acc[a][b][4 * grp + 1], acc[a][b][4 * grp + 2],
                           acc[a][b][4 * grp + 3]};
        *reinterpret_cast<floatx4*>(ws + (lane & 31) * LD + a * 32 + 8 * grp + 4 * (lane >> 5)) = v;
      }
    // the wave reads back only what it wrote: LDS accesses of a wave stay in order
#pragma unroll
    for (int q = 0; q < 32 / CPI; ++q) {
      const int j = q * CPI + lane / LPC, i = 4 * (lane % LPC);
      const floatx4 v = *reinterpret_cast<const floatx4*>(ws + j * LD + i);
      const int64_t gi = s.i0 + wm * RW + i, gj = s.j0 + wn * 64 + b * 32 + j;
      *reinterpret_cast<floatx4*>(xo + gi + gj * s.sc) = v;
    }
  }
}

// bf16x3 (NP = 3) double-buffers the LDS slabs: while the products of slab s
// run from one buffer, slab s + 1 is split and stored into the other and the
// global loads of slab s + 2 are in flight; one barrier per slab, and the
// steady-state loop body is a single basic block (the look-ahead slab index
// is clamped to the last slab instead of branching), so that the compiler can
// interleave the split arithmetic with the matrix products.  bf16x5 and
// bf16x6 need 1.25x and 1.5x the LDS per buffer and keep a single buffer
// with two barriers.
// SCALED: the X operands are multiplied by the first step's 1/||Delta||_F.
template <int MODE, int NP, int LAYOUT, bool SCALED, bool SAME = false>
__device__ __forceinline__ void bf16_tile(const GemmArgs& g, const Task& task,
                                          __bf16 (*Ap)[SplitParts<NP>::a][kBM][kLdsK],
                                          __bf16 (*Bp)[SplitParts<NP>::b][kBN][kLdsK]) {
  constexpr int kNa = SplitParts<NP>::a, kNb = SplitParts<NP>::b, NB = SplitParts<NP>::nb;
  // only X operands carry a scale (Gram: both, Update: A)
  constexpr bool SA = SCALED && MODE != kPoly;
  constexpr bool SB = SCALED && MODE == kGram;
  const GemmSetup s = gemm_setup<MODE>(g, task);
  // SAME: a diagonal tile of a symmetric product, whose two operand panels
  // coincide -- loaded, split and stored once, read as both operands
  auto bpl = [&](int buf) -> __bf16 (*)[kBN][kLdsK] {
    if constexpr (SAME) return Ap[buf];
    else return Bp[buf];
  };
  floatx16 acc[2][2];
  gemm_acc_init<MODE>(g, s, acc);

  const int nslab = (s.k_end - s.k_begin + kBK2 - 1) / kBK2;
  const int klast = s.k_begin + (nslab - 1) * kBK2;
  Slab32 ra, rb;
  if (nslab > 0) {
  load_operand<MODE, LAYOUT>(s.A, s.k_begin, s.i0, ra);
  if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, s.k_begin, s.j0, rb);
  if (NB == 2) {
    // Registers hold two slabs in flight: at the top of the products of slab
    // sl, slab sl + 1 is in (ra1, rb1) and slab sl + 2 in (ra, rb).  Each
    // iteration splits and stores the first into the idle LDS buffer and
    // reloads its registers with slab sl + 3, so a load has about two slabs of
    // products to land.  The loop is unrolled by two so that the register
    // roles are static.
    auto kat = [&](int sl) { return min(s.k_begin + sl * kBK2, klast); };
    Slab32 ra1, rb1;
    load_operand<MODE, LAYOUT>(s.A, kat(1), s.i0, ra1);
    if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, kat(1), s.j0, rb1);
    store_operand<MODE, LAYOUT, kNa, SA>(ra, Ap[0], s.A.scale);
    if constexpr (!SAME) store_operand<MODE, LAYOUT, kNb, SB>(rb, Bp[0], s.B.scale);
    load_operand<MODE, LAYOUT>(s.A, kat(2), s.i0, ra);
    if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, kat(2), s.j0, rb);
    __syncthreads();
    int sl = 0;
    for (; sl + 2 < nslab; sl += 2) {
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 0, acc);
      store_operand<MODE, LAYOUT, kNa, SA>(ra1, Ap[1], s.A.scale);
      if constexpr (!SAME) store_operand<MODE, LAYOUT, kNb, SB>(rb1, Bp[1], s.B.scale);
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 16, acc);
      load_operand<MODE, LAYOUT>(s.A, kat(sl + 3), s.i0, ra1);
      if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, kat(sl + 3), s.j0, rb1);
      __syncthreads();
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[1], bpl(1), 0, acc);
      store_operand<MODE, LAYOUT, kNa, SA>(ra, Ap[0], s.A.scale);
      if constexpr (!SAME) store_operand<MODE, LAYOUT, kNb, SB>(rb, Bp[0], s.B.scale);
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[1], bpl(1), 16, acc);
      load_operand<MODE, LAYOUT>(s.A, kat(sl + 4), s.i0, ra);
      if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, kat(sl + 4), s.j0, rb);
      __syncthreads();
    }
    // one or two slabs remain: slab sl in buffer 0, slab sl + 1 in (ra1, rb1)
    int last = 0;
    if (sl + 1 < nslab) {
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 0, acc);
      store_operand<MODE, LAYOUT, kNa, SA>(ra1, Ap[1], s.A.scale);
      if constexpr (!SAME) store_operand<MODE, LAYOUT, kNb, SB>(rb1, Bp[1], s.B.scale);
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 16, acc);
      __syncthreads();
      last = 1;
    }
    mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[last], bpl(last), 0, acc);
    mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[last], bpl(last), 16, acc);
  } else {
    for (int sl = 0; sl < nslab; ++sl) {
      __syncthreads();
      store_operand<MODE, LAYOUT, kNa, SA>(ra, Ap[0], s.A.scale);
      if constexpr (!SAME) store_operand<MODE, LAYOUT, kNb, SB>(rb, Bp[0], s.B.scale);
      __syncthreads();
      const int k1 = min(s.k_begin + (sl + 1) * kBK2, klast);
      load_operand<MODE, LAYOUT>(s.A, k1, s.i0, ra);
      if constexpr (!SAME) load_operand<MODE, LAYOUT>(s.B, k1, s.j0, rb);
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 0, acc);
      mfma_substep<kNa, kNb, 2, 2, kBM>(Ap[0], bpl(0), 16, acc);
    }
  }
  }
  if constexpr (MODE == kUpdate && LAYOUT == kFast)
    store_update_colmajor<2, 2>(g, s, acc, reinterpret_cast<float*>(&Ap[0][0][0][0]));
  else
    gemm_epilogue<MODE, 2, 2>(g, s, task, acc, &Ap[0][0][0][0]);
}

// 128 x 128 tiles: the interior tiles (kFast; the diagonal tiles of the
// symmetric products stage their one operand panel once) or the ragged ones
// (kGeneric).
template <int MODE, int NP, int LAYOUT, bool SCALED>
__global__ void __launch_bounds__(kGemmThreads, 2) gemm_bf16_kernel(GemmArgs g) {
  constexpr int NB = SplitParts<NP>::nb;
  typedef __bf16 APlanes[SplitParts<NP>::a][kBM][kLdsK];
  typedef __bf16 BPlanes[SplitParts<NP>::b][kBM][kLdsK];
  const Task task = g.tasks[blockIdx.x];
  if (task.mat < 0 || (g.only_active && !g.sc[task.mat].active)) return;
  auto run = [&](APlanes* Ap, BPlanes* Bp) {
    if constexpr (LAYOUT == kFast && MODE != kUpdate) {
      const bool same = task.tm == task.tn && (MODE == kPoly || !g.bin);
      if (same) bf16_tile<MODE, NP, kFast, SCALED, true>(g, task, Ap, Bp);
      else bf16_tile<MODE, NP, kFast, SCALED>(g, task, Ap, Bp);
    } else {
      bf16_tile<MODE, NP, LAYOUT, SCALED>(g, task, Ap, Bp);
    }
  };
  if constexpr (MODE == kUpdate) {
    // one block for the operand planes and, after the products, the staging
    // of the output tile
    constexpr size_t kPlanes = NB * (sizeof(APlanes) + sizeof(BPlanes));
    constexpr size_t kStage = stage_floats<2>(kGemmThreads / 64) * sizeof(float);
    __shared__ __attribute__((aligned(16))) char lds[kPlanes > kStage ? kPlanes : kStage];
    run(reinterpret_cast<APlanes*>(lds), reinterpret_cast<BPlanes*>(lds + NB * sizeof(APlanes)));
  } else {
    __shared__ __attribute__((aligned(16))) APlanes Ap[NB];
    __shared__ __attribute__((aligned(16))) BPlanes Bp[NB];
    run(Ap, Bp);
  }
}

// 256 x 256 block tiles of the update products (interior tiles of the
// column-major iterates; the planner lists 256 x 256 tiles for the updates
// alone), so that every fp32 operand value staged through LDS feeds twice as
// many products as on 128 x 128 tiles -- half the global loads, splits, LDS
// writes and barriers per product.  bf16x3 and bf16x5 double-buffer LDS (the
// whole 160 KB of the CU: 2 buffers of 2 + 2 planes of 80-byte rows, or of
// 3 + 2 planes of 64-byte rows) on 1024 threads (gemm_bf16_big16_kernel);
// bf16x6 keeps one buffer of 3 + 3 planes (120 KB) and two barriers per slab,
// on 512 threads in 8 waves of 128 x 64 (2 x 4) (gemm_bf16_big_kernel).
constexpr int kBig = 256;
constexpr int kBigThreads = 512;

// LDS of the 256 x 256 kernel: bf16x3 double-buffers 80-byte rows (2 x 2 x 2
// planes of 256 rows: 160 KB); bf16x5 double-buffers 64-byte rows (2 x (3 + 2)
// planes: 160 KB; with 80-byte rows one buffer only, two barriers per slab:
// its updates took 2.6x the time of a bf16x3 update for 1.67x the products);
// bf16x6 keeps one buffer of 80-byte rows.
template <int NP>
struct BigLds {
  static constexpr int nb = NP == 6 ? 1 : 2;            // LDS buffers
  static constexpr int lk = NP == 5 ? kBK2 : kLdsK;     // row pitch (bf16 elements)
};

template <int MODE, int NP, bool SCALED>
__device__ __forceinline__ void bf16_big_tile(const GemmArgs& g, const Task& task,
                                              __bf16 (*Ap)[SplitParts<NP>::a][kBig][BigLds<NP>::lk],
                                              __bf16 (*Bp)[SplitParts<NP>::b][kBig][BigLds<NP>::lk]) {
  static_assert(MODE == kUpdate, "256 x 256 tiles serve the update products");
  static_assert(BigLds<NP>::nb == 1, "the double-buffered updates run on gemm_bf16_big16_kernel");
  constexpr int LAYOUT = kFast;
  constexpr int kNa = SplitParts<NP>::a, kNb = SplitParts<NP>::b, LK = BigLds<NP>::lk;
  constexpr bool SA = SCALED;  // the X operand carries the first step's scale
  constexpr bool SB = false;
  const GemmSetup s = gemm_setup<MODE, kBig>(g, task);
  floatx16 acc[4][2];
  gemm_acc_init<MODE, 4, 4>(g, s, acc);

  const int nslab = (s.k_end - s.k_begin + kBK2 - 1) / kBK2;
  if (nslab > 0) {
    const int klast = s.k_begin + (nslab - 1) * kBK2;
    auto kat = [&](int sl) { return min(s.k_begin + sl * kBK2, klast); };
    Slab32 ra, rb;
    load_operand<MODE, LAYOUT, kBig, LK>(s.A, s.k_begin, s.i0, ra);
    load_operand<MODE, LAYOUT, kBig, LK>(s.B, s.k_begin, s.j0, rb);
    for (int sl = 0; sl < nslab; ++sl) {
      __syncthreads();
      store_operand<MODE, LAYOUT, kNa, SA, kBig, LK>(ra, Ap[0], s.A.scale);
      store_operand<MODE, LAYOUT, kNb, SB, kBig, LK>(rb, Bp[0], s.B.scale);
      __syncthreads();
      load_operand<MODE, LAYOUT, kBig, LK>(s.A, kat(sl + 1), s.i0, ra);
      load_operand<MODE, LAYOUT, kBig, LK>(s.B, kat(sl + 1), s.j0, rb);
      mfma_substep<kNa, kNb, 4, 4, kBig, LK>(Ap[0], Bp[0], 0, acc);
      mfma_substep<kNa, kNb, 4, 4, kBig, LK>(Ap[0], Bp[0], 16, acc);
    }
  }
  store_update_colmajor<4, 4>(g, s, acc, reinterpret_cast<float*>(&Ap[0][0][0][0]));
}

template <int MODE, int NP, bool SCALED>
__global__ void __launch_bounds__(kBigThreads, 1) gemm_bf16_big_kernel(GemmArgs g) {
  constexpr int NB = BigLds<NP>::nb;
  typedef __bf16 APlanes[SplitParts<NP>::a][kBig][BigLds<NP>::lk];
  typedef __bf16 BPlanes[SplitParts<NP>::b][kBig][BigLds<NP>::lk];
  const Task task = g.tasks[blockIdx.x];
  if (task.mat < 0 || (g.only_active && !g.sc[task.mat].active)) return;
  // one block for the operand planes and, after the products, the staging
  // of the output tile
  constexpr size_t kPlanes = NB * (sizeof(APlanes) + sizeof(BPlanes));
  constexpr size_t kStage = stage_floats<4>(kBigThreads / 64) * sizeof(float);
  __shared__ __attribute__((aligned(16))) char lds[kPlanes > kStage ? kPlanes : kStage];
  bf16_big_tile<MODE, NP, SCALED>(g, task, reinterpret_cast<APlanes*>(lds),
                                  reinterpret_cast<BPlanes*>(lds + NB * sizeof(APlanes)));
}

// The bf16x3 and bf16x5 updates' 256 x 256 tiles run on 1024 threads: 16 waves
// of 64 x 64 (4 x 4), four per SIMD instead of two, each thread staging 8
// values of each operand per slab (one slab in flight in registers), the same
// double-buffered LDS as the 512-thread kernel and the same products in the
// same order per output element (bit for bit the same results).  The two
// extra waves per SIMD hide more of the operand latency: update launches 3%
// (109.5M workload) to 5% (341M) shorter.  bf16x6 keeps the 512-thread kernel
// (one LDS buffer).
constexpr int kBig16Threads = 1024;

// 8 values of an i-contiguous operand: row i0 + t % ROWS, k = k0 + 8 (t / ROWS) .. +7
template <int ROWS>
__device__ __forceinline__ void slab16_load_icontig(const Operand& op, int k0, int i0, floatx4 (&r)[2]) {
  const int t = threadIdx.x;
  const int bytes = 4 * ((op.K - 1) * (int)op.s_k + (op.I - 1) * (int)op.s_i + 1);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(op.base), (short)0, bytes, kBufferFlags);
  const int kb = k0 + 8 * __builtin_amdgcn_readfirstlane(t / ROWS);
  const int vo = 4 * (i0 + t % ROWS);
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      r[q][e] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(rs, vo, 4 * (kb + 4 * q + e) * (int)op.s_k, 0));
}

// Split the thread's 8 values into NS bf16 parts (as slab32_store) and store
// each part plane as one 16-byte row segment.
template <int NS, bool SCALED, int ROWS, int LK>
__device__ __forceinline__ void slab16_store(const floatx4 (&r)[2], __bf16 (*planes)[ROWS][LK], float scale) {
  const int t = threadIdx.x;
  const int i = t % ROWS, c = t / ROWS;
  bf16x8 part[NS];
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    floatx2 x = {r[e / 4][e % 4], r[e / 4][e % 4 + 1]};
    if (SCALED) x *= scale;
#pragma unroll
    for (int p = 0; p < NS; ++p) {
      const bf16x2 h = __builtin_convertvector(x, bf16x2);
      part[p][e] = h[0];
      part[p][e + 1] = h[1];
      if (p + 1 < NS) x -= __builtin_convertvector(h, floatx2);
    }
  }
#pragma unroll
  for (int p = 0; p < NS; ++p) *reinterpret_cast<bf16x8*>(&planes[p][i][lds_chunk<LK>(i, c)]) = part[p];
}

template <int NP, bool SCALED>
__global__ void __launch_bounds__(kBig16Threads, 1) gemm_bf16_big16_kernel(GemmArgs g) {
  constexpr int MODE = kUpdate;
  static_assert(BigLds<NP>::nb == 2, "double-buffered LDS");
  constexpr int kNa = SplitParts<NP>::a, kNb = SplitParts<NP>::b, LK = BigLds<NP>::lk;
  typedef __bf16 APlanes[kNa][kBig][LK];
  typedef __bf16 BPlanes[kNb][kBig][LK];
  constexpr size_t kPlanes = 2 * (sizeof(APlanes) + sizeof(BPlanes));
  constexpr size_t kStage = stage_floats<2>(kBig16Threads / 64) * sizeof(float);
  __shared__ __attribute__((aligned(16))) char lds[kPlanes > kStage ? kPlanes : kStage];
  const Task task = g.tasks[blockIdx.x];
  if (task.mat < 0 || (g.only_active && !g.sc[task.mat].active)) return;
  APlanes* Ap = reinterpret_cast<APlanes*>(lds);
  BPlanes* Bp = reinterpret_cast<BPlanes*>(lds + 2 * sizeof(APlanes));
  const GemmSetup s = gemm_setup<MODE, kBig>(g, task);
  floatx16 acc[2][2];
  gemm_acc_init<MODE, 2, 4>(g, s, acc);
  const int nslab = (s.k_end - s.k_begin + kBK2 - 1) / kBK2;
  if (nslab > 0) {
    const int klast = s.k_begin + (nslab - 1) * kBK2;
    auto kat = [&](int sl) { return min(s.k_begin + sl * kBK2, klast); };
    floatx4 ra[2], rb[2];
    slab16_load_icontig<kBig>(s.A, s.k_begin, s.i0, ra);
    slab16_load_icontig<kBig>(s.B, s.k_begin, s.j0, rb);
    slab16_store<kNa, SCALED, kBig, LK>(ra, Ap[0], s.A.scale);
    slab16_store<kNb, false, kBig, LK>(rb, Bp[0], s.B.scale);
    slab16_load_icontig<kBig>(s.A, kat(1), s.i0, ra);
    slab16_load_icontig<kBig>(s.B, kat(1), s.j0, rb);
    __syncthreads();
    for (int sl = 0; sl + 1 < nslab; ++sl) {
      const int cur = sl & 1;
      mfma_substep<kNa, kNb, 2, 4, kBig, LK>(Ap[cur], Bp[cur], 0, acc);
      slab16_store<kNa, SCALED, kBig, LK>(ra, Ap[cur ^ 1], s.A.scale);
      slab16_store<kNb, false, kBig, LK>(rb, Bp[cur ^ 1], s.B.scale);
      mfma_substep<kNa, kNb, 2, 4, kBig, LK>(Ap[cur], Bp[cur], 16, acc);
      slab16_load_icontig<kBig>(s.A, kat(sl + 2), s.i0, ra);
      slab16_load_icontig<kBig>(s.B, kat(sl + 2), s.j0, rb);
      __syncthreads();
    }
    const int last = (nslab - 1) & 1;
    mfma_substep<kNa, kNb, 2, 4, kBig, LK>(Ap[last], Bp[last], 0, acc);
    mfma_substep<kNa, kNb, 2, 4, kBig, LK>(Ap[last], Bp[last], 16, acc);
  }
  store_update_colmajor<2, 4>(g, s, acc, reinterpret_cast<float*>(lds));
}

// The per-matrix decisions of a phase end without a Gram launch (kActStop
// only: nothing to sum).
__global__ void gram_norm_final_kernel(const MatInfo* __restrict__ mats, const double* __restrict__ part,
                                       MatScalars* __restrict__ sc, int n_mat, NormArgs a) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= n_mat) return;
  if (a.only_active && !sc[m].active) return;
  norm_decide(mats[m], part, sc[m], a);
}

// The scale of a correction (sigma_bar).  mode 0: <Q, Delta>_F / r, the mean
// singular value (tr is <Q, Delta>_F); 1: ||Delta||_F / sqrt(r), their RMS;
// 2: sqrt(rows / cols) of the tensor as stored (Muon's sqrt(fan_out / fan_in)).
__device__ __forceinline__ void set_sigma(MatScalars& o, const MatInfo& mi, double tr, int mode) {
  if (o.flags & kFlagNonfinite) o.sigma_bar = __builtin_nanf("");
  else if (o.flags & kFlagZero) o.sigma_bar = 0.f;
  else if (mode == 0) o.sigma_bar = (float)(tr / mi.n);
  else if (mode == 1) o.sigma_bar = (float)((double)o.fro / sqrt((double)mi.n));
  else o.sigma_bar = (float)(mi.wide ? sqrt((double)mi.n / mi.m) : sqrt((double)mi.m / mi.n));
}

// <Q, Delta>_F partial per chunk of a corrected matrix (both in the
// workspace layout: chunk_ws maps the chunk's elements; groups of 4 are
// contiguous when c.vec).  The last chunk of a matrix to arrive (counted in
// mat_cnt) adds the matrix's partials in a fixed order (that of
// block_sum_range) and sets its sigma_bar = <Q, Delta>_F / r.
__global__ void __launch_bounds__(kStreamThreads)
trace_kernel(const Chunk* __restrict__ chunks, const int* __restrict__ idx, const MatInfo* __restrict__ mats,
             MatScalars* __restrict__ sc, const float* __restrict__ x0, const float* __restrict__ x1,
             const float* __restrict__ delta, double* __restrict__ part_tr, int* __restrict__ mat_cnt, int steps_lo,
             int steps_hi) {
  __shared__ double red[4];
  __shared__ int last;
  const int ci = idx ? idx[blockIdx.x] : (int)blockIdx.x;
  const Chunk c = chunks[ci];
  const int st = sc[c.mat].steps;
  if (st < steps_lo || st > steps_hi) return;
  const float* q = sc[c.mat].qbuf ? x1 : x0;
  double s = 0.0;
  int done = 0;
  if (c.vec) {
    const int nv = c.count / 4;
    for (int v = threadIdx.x; v < nv; v += kStreamThreads) {
      const int64_t o = chunk_ws(c, 4 * v);
      const floatx4 a = *reinterpret_cast<const floatx4*>(q + o);
      const floatx4 d = *reinterpret_cast<const floatx4*>(delta + o);
      s += (double)a[0] * d[0] + (double)a[1] * d[1] + (double)a[2] * d[2] + (double)a[3] * d[3];
    }
    done = nv * 4;
  }
  for (int i = done + threadIdx.x; i < c.count; i += kStreamThreads) {
    const int64_t o = chunk_ws(c, i);
    s += (double)q[o] * delta[o];
  }
  s = block_sum256(s, red);
  const MatInfo& mi = mats[c.mat];
  if (threadIdx.x == 0) {
    partial_store(part_tr + ci, s);
    last = arrive(mat_cnt + c.mat, mi.chunk_end - mi.chunk_begin);
  }
  __syncthreads();
  if (!last) return;
  double t = 0.0;
  for (int x = mi.chunk_begin + (int)threadIdx.x; x < mi.chunk_end; x += 256) t += partial_load(part_tr + x);
  t = block_sum256(t, red);
  if (threadIdx.x == 0) set_sigma(sc[c.mat], mi, t, 0);
}

// The closed-form scales (modes 1 and 2 of set_sigma), one block per matrix.
__global__ void __launch_bounds__(256)
sigma_kernel(const MatInfo* __restrict__ mats, MatScalars* __restrict__ sc, int n_mat, int mode, int cls,
             int steps_lo, int steps_hi) {
  const int m = blockIdx.x;
  const MatInfo mi = mats[m];
  if (cls >= 0 && mi.sched != cls) return;
  if (sc[m].steps < steps_lo || sc[m].steps > steps_hi) return;
  if (threadIdx.x == 0) set_sigma(sc[m], mi, 0.0, mode);
}

// One element of the write-back: D = f p;  B <- mu B + D;  theta <- theta - lr (D + mu B)
// (heavy_ball: theta <- theta - lr B; target_update: B was updated by the
// reduction and theta <- theta - lr D).
__device__ __forceinline__ void finish_one(float* __restrict__ theta, float* __restrict__ mom, int64_t e, float d,
                                           float lr, float mu, int heavy_ball, int target_update) {
  if (target_update) {
    theta[e] = theta[e] - lr * d;
  } else {
    const float bn = mu * mom[e] + d;
    mom[e] = bn;
    theta[e] = theta[e] - lr * (heavy_ball ? bn : d + mu * bn);
  }
}

__device__ __forceinline__ void finish_quad(float* __restrict__ theta, float* __restrict__ mom, int64_t e,
                                            const floatx4& d, float lr, float mu, int heavy_ball, int target_update) {
  floatx4 t = *reinterpret_cast<const floatx4*>(theta + e);
  if (target_update) {
#pragma unroll
    for (int r = 0; r < 4; ++r) t[r] = t[r] - lr * d[r];
  } else {
    floatx4 b = *reinterpret_cast<const floatx4*>(mom + e);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float bn = mu * b[r] + d[r];
      b[r] = bn;
      t[r] = t[r] - lr * (heavy_ball ? bn : d[r] + mu * bn);
    }
    *reinterpret_cast<floatx4*>(mom + e) = b;
  }
  *reinterpret_cast<floatx4*>(theta + e) = t;
}

// The write-back of the corrected tensors (Algorithm 2): D = f P with P = Q
// and f = alpha sigma_bar (clip variants: P is their correction, already
// scaled, and f = 1).  A tile chunk reads its column-major P through LDS.
__global__ void __launch_bounds__(kStreamThreads)
finish_kernel(const Chunk* __restrict__ chunks, const int* __restrict__ idx, const MatScalars* __restrict__ sc,
              const float* __restrict__ x0, const float* __restrict__ x1, const float* __restrict__ dclip,
              float* __restrict__ theta, float* __restrict__ mom, float alpha, float lr, float mu, int heavy_ball,
              int target_update, int clip, int steps_lo, int steps_hi) {
  __shared__ TileLds tl;
  const Chunk c = chunks[idx ? idx[blockIdx.x] : blockIdx.x];
  const MatScalars s = sc[c.mat];
  if (s.steps < steps_lo || s.steps > steps_hi) return;
  const float* q = clip ? dclip : (s.qbuf ? x1 : x0);
  float f = clip ? 1.f : alpha * s.sigma_bar;
  if (s.flags & kFlagZero) f = 0.f;
  if (c.rows) {
    const int TR = c.rows, TC = c.cols;
    for (int it = threadIdx.x; it < TC * (kTileRows / 4); it += kStreamThreads) {
      const int cc = it / (kTileRows / 4), r = 4 * (it % (kTileRows / 4));
      if (r >= TR) continue;
      const float* src = q + c.ws + (int64_t)cc * c.ws_ld + r;
      if (c.vec) {
        const floatx4 v = *reinterpret_cast<const floatx4*>(src);
        tl[r][cc] = v[0]; tl[r + 1][cc] = v[1]; tl[r + 2][cc] = v[2]; tl[r + 3][cc] = v[3];
      } else {
        for (int k = 0; k < 4 && r + k < TR; ++k) tl[r + k][cc] = src[k];
      }
    }
    __syncthreads();
    for (int it = threadIdx.x; it < TR * (kTileCols / 4); it += kStreamThreads) {
      const int rr = it / (kTileCols / 4), col = 4 * (it % (kTileCols / 4));
      if (col >= TC) continue;
      const int64_t e = c.src + (int64_t)rr * c.src_ld + col;
      if (c.vec) {
        const floatx4 d = {f * tl[rr][col], f * tl[rr][col + 1], f * tl[rr][col + 2], f * tl[rr][col + 3]};
        finish_quad(theta, mom, e, d, lr, mu, heavy_ball, target_update);
      } else {
        for (int k = 0; k < 4 && col + k < TC; ++k)
          finish_one(theta, mom, e + k, f * tl[rr][col + k], lr, mu, heavy_ball, target_update);
      }
    }
    return;
  }
  int done = 0;
  if (c.vec) {
    const int nv = c.count / 4;
    for (int v = threadIdx.x; v < nv; v += kStreamThreads) {
      const floatx4 qq = *reinterpret_cast<const floatx4*>(q + c.ws + 4 * v);
      finish_quad(theta, mom, c.src + 4 * v, f * qq, lr, mu, heavy_ball, target_update);
    }
    done = nv * 4;
  }
  for (int i = done + threadIdx.x; i < c.count; i += kStreamThreads)
    finish_one(theta, mom, c.src + i, f * q[c.ws + i], lr, mu, heavy_ball, target_update);
}

// Clip variants, first half: E = Delta - sigma_bar Q in place of Delta, Q
// copied aside, and the chunk partials of ||E||^2 for the second iteration
// (all in the workspace layout).
__global__ void __launch_bounds__(kStreamThreads)
clip_prep_kernel(const Chunk* __restrict__ chunks, const MatScalars* __restrict__ sc, const float* __restrict__ x0,
                 const float* __restrict__ x1, float* __restrict__ delta, float* __restrict__ qcopy,
                 double* __restrict__ part_sq) {
  __shared__ double red[4];
  const Chunk c = chunks[blockIdx.x];
  const MatScalars s = sc[c.mat];
  const float* q = s.qbuf ? x1 : x0;
  const float sb = (s.flags & kFlagInput) ? 0.f : s.sigma_bar;
  double sq = 0.0;
  for (int i = threadIdx.x; i < c.count; i += kStreamThreads) {
    const int64_t o = chunk_ws(c, i);
    const float qv = q[o];
    const float ev = delta[o] - sb * qv;
    delta[o] = ev;
    qcopy[o] = qv;
    sq += (double)ev * ev;
  }
  sq = block_sum256(sq, red);
  if (threadIdx.x == 0) part_sq[blockIdx.x] = sq;
}

// Clip variants, the correction in the workspace layout, in place of E:
// clip_high D = alpha ((E - |E|) / 2 + sigma_bar Q), clip_low alpha ((E + |E|) / 2
// + sigma_bar Q), with E = Delta - sigma_bar Q (delta), |E| = Q (Q2^T E) (x0)
// and Q (qcopy).
__global__ void __launch_bounds__(kStreamThreads)
clip_compose_kernel(const Chunk* __restrict__ chunks, const MatScalars* __restrict__ sc, const float* __restrict__ x0,
                    const float* __restrict__ qcopy, float* __restrict__ delta, float alpha, int clip) {
  const Chunk c = chunks[blockIdx.x];
  const MatScalars s = sc[c.mat];
  const float sg = clip == 1 ? -0.5f : 0.5f;
  const float sb = s.sigma_bar;
  const float al = (s.flags & kFlagZero) ? 0.f : alpha;
  for (int i = threadIdx.x; i < c.count; i += kStreamThreads) {
    const int64_t o = chunk_ws(c, i);
    delta[o] = al * (0.5f * delta[o] + sg * x0[o] + sb * qcopy[o]);
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

hipError_t launch_reduce(const DevTables& t, const StepArgs& a, hipStream_t st) {
  if (t.n_chunks == 0) return hipSuccess;
  const float inv_k = 1.0f / (float)a.K;
  if (a.worker_dtype == 0)
    hipLaunchKernelGGL(reduce_kernel<0>, dim3(t.n_chunks), dim3(kStreamThreads), 0, st, t.chunks,
                       a.theta, a.mom, t.delta, t.part_sq, a.workers, a.K, inv_k, a.lr, a.mu, a.heavy_ball,
                       a.target_update);
  else
    hipLaunchKernelGGL(reduce_kernel<1>, dim3(t.n_chunks), dim3(kStreamThreads), 0, st, t.chunks,
                       a.theta, a.mom, t.delta, t.part_sq, a.workers, a.K, inv_k, a.lr, a.mu, a.heavy_ball,
                       a.target_update);
  return hipGetLastError();
}

hipError_t launch_fro(const DevTables& t, const FroArgs& a, hipStream_t st) {
  if (t.n_mat == 0) return hipSuccess;
  hipLaunchKernelGGL(fro_kernel, dim3(t.n_mat), dim3(256), 0, st, t.mats, t.part_sq, t.scalars, t.n_mat, a);
  return hipGetLastError();
}

// segment 0: interior tiles; segment 1: ragged tiles (bounds-checked loads)
template <int MODE, int NP, bool SCALED>
static void launch_bf16_segments(const Task* tasks, const int* off, const int* cnt, const GemmArgs& g0,
                                 hipStream_t st) {
  GemmArgs g = g0;
  const dim3 block(kGemmThreads);
  if (cnt[0]) {
    g.tasks = tasks + off[0];
    hipLaunchKernelGGL((gemm_bf16_kernel<MODE, NP, kFast, SCALED>), dim3(cnt[0]), block, 0, st, g);
  }
  if (cnt[1]) {
    g.tasks = tasks + off[1];
    hipLaunchKernelGGL((gemm_bf16_kernel<MODE, NP, kGeneric, SCALED>), dim3(cnt[1]), block, 0, st, g);
  }
}

// The 256 x 256 interior tiles, then the 128 x 128 tiles left over (for lists
// without 256 x 256 tiles this is the plain 128 x 128 cover).
template <int MODE, int NP, bool SCALED>
static void launch_big_cover(const TaskList& L, const GemmArgs& g0, hipStream_t st) {
  GemmArgs g = g0;
  const dim3 block(kBigThreads);
  // (the planner lists 256 x 256 tiles for the update products only)
  if constexpr (MODE == kUpdate) {
    if (L.big_cnt) {
      g.tasks = L.tasks + L.big_off;
      if constexpr (NP == 3 || NP == 5)
        hipLaunchKernelGGL((gemm_bf16_big16_kernel<NP, SCALED>), dim3(L.big_cnt), dim3(kBig16Threads), 0, st, g);
      else
        hipLaunchKernelGGL((gemm_bf16_big_kernel<MODE, NP, SCALED>), dim3(L.big_cnt), block, 0, st, g);
    }
  }
  launch_bf16_segments<MODE, NP, SCALED>(L.tasks, L.rem_off, L.rem_cnt, g0, st);
}

// The first step's X operands carry the 1/||Delta||_F pre-scaling (Poly reads
// only Gram outputs and never does).
template <int MODE, int NP>
static void launch_bf16(const TaskList& L, const GemmArgs& g, hipStream_t st) {
  if (MODE != kPoly && g.first) launch_big_cover<MODE, NP, MODE != kPoly>(L, g, st);
  else launch_big_cover<MODE, NP, false>(L, g, st);
}

template <int MODE>
static void launch_mode(const TaskList& L, const GemmArgs& g0, int arith, hipStream_t st) {
  if (arith == kArithFp32) {
    GemmArgs g = g0;
    g.tasks = L.tasks;
    const int n = L.seg_cnt[0] + L.seg_cnt[1];
    if (n) hipLaunchKernelGGL(gemm_f32_kernel<MODE>, dim3(n), dim3(kGemmThreads), 0, st, g);
  } else if (arith == kArithBf16x6) {
    launch_bf16<MODE, 6>(L, g0, st);
  } else if (MODE == kUpdate && arith == kArithBf16x5) {
    launch_bf16<MODE, 5>(L, g0, st);
  } else {
    launch_bf16<MODE, 3>(L, g0, st);
  }
}

hipError_t launch_gemm(const DevTables& t, int mode, const PolarStep& p, hipStream_t st) {
  GemmArgs g;
  g.mats = t.mats;
  g.sc = t.scalars;
  g.xin = p.xin;
  g.xin_alt = p.xin_alt;
  g.bin = p.bin;
  g.xout = p.xout;
  g.gram = t.gram;
  g.poly = t.poly;
  g.gpart = t.gpart;
  g.split_cnt = t.split_cnt;
  g.mat_cnt = t.mat_cnt;
  g.sc_out = t.scalars;
  g.part_norm = t.part_norm;
  g.norm_mode = mode == kGram ? p.norm_mode : -1;
  g.na = p.norm;
  g.coef = t.coef;
  g.step = p.step;
  g.n_steps = t.n_steps;
  g.first = p.first;
  g.only_active = p.only_active;
  g.tasks = nullptr;
  if (mode == kGram) launch_mode<kGram>(t.gram_list, g, p.arith, st);
  else if (mode == kPoly) launch_mode<kPoly>(t.poly_list, g, p.arith, st);
  else launch_mode<kUpdate>(t.update_list, g, p.arith, st);
  return hipGetLastError();
}

hipError_t launch_gram_norm(const DevTables& t, const NormArgs& a, hipStream_t st) {
  if (t.n_mat == 0) return hipSuccess;
  hipLaunchKernelGGL(gram_norm_final_kernel, dim3((t.n_mat + 63) / 64), dim3(64), 0, st, t.mats, t.part_norm,
                     t.scalars, t.n_mat, a);
  return hipGetLastError();
}

hipError_t launch_scale(const DevTables& t, const StepArgs& a, hipStream_t st) {
  const int n = t.chunk_idx ? t.n_chunk_idx : t.n_iso_chunks;
  if (n == 0) return hipSuccess;
  if (a.scale == 0)
    hipLaunchKernelGGL(trace_kernel, dim3(n), dim3(kStreamThreads), 0, st, t.chunks, t.chunk_idx, t.mats,
                       t.scalars, t.x[0], t.x[1], t.delta, t.part_tr, t.mat_cnt, a.steps_lo, a.steps_hi);
  else
    hipLaunchKernelGGL(sigma_kernel, dim3(t.n_mat), dim3(256), 0, st, t.mats, t.scalars, t.n_mat, a.scale, t.cls,
                       a.steps_lo, a.steps_hi);
  return hipGetLastError();
}

hipError_t launch_finish(const DevTables& t, const StepArgs& a, hipStream_t st) {
  const int n = t.chunk_idx ? t.n_chunk_idx : t.n_iso_chunks;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(finish_kernel, dim3(n), dim3(kStreamThreads), 0, st, t.chunks, t.chunk_idx, t.scalars,
                     t.x[0], t.x[1], t.delta, a.theta, a.mom, a.alpha, a.lr, a.mu, a.heavy_ball, a.target_update,
                     a.clip, a.steps_lo, a.steps_hi);
  return hipGetLastError();
}

hipError_t launch_clip_compose(const DevTables& t, const StepArgs& a, hipStream_t st) {
  if (t.n_iso_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(clip_compose_kernel, dim3(t.n_iso_chunks), dim3(kStreamThreads), 0, st, t.chunks, t.scalars,
                     t.x[0], t.x2, t.delta, a.alpha, a.clip);
  return hipGetLastError();
}

}  // namespace isoloco

namespace isoloco {
hipError_t launch_clip_prep(const DevTables& t, hipStream_t st) {
  if (t.n_iso_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(clip_prep_kernel, dim3(t.n_iso_chunks), dim3(kStreamThreads), 0, st, t.chunks, t.scalars,
                     t.x[0], t.x[1], t.delta, t.x2, t.part_sq);
  return hipGetLastError();
}
}  // namespace isoloco
