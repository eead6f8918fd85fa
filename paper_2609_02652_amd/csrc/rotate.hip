// Activation rotation for gfx950 (§2.3 "The kernel": a separate kernel rotates
// the activation before the matvec; §6 "The rotated basis and the shared-memory
// wall": weights live in the rotated basis, so every consumer rotates).
//
// For K = n·m with n = 2^k the largest power of two dividing K, block b of n
// consecutive coordinates becomes n^(-1/2) · H_n · (s ⊙ x), with
// H_n[i][j] = (−1)^popcount(i & j) (Sylvester order) and s the caller's ±1
// signs.  The transform is a product of k butterfly stages, one per index
// bit; stages over distinct bits commute, so they may be taken in any order.
//
// Geometry.  A workgroup owns a segment of S = max(n, 2048) coordinates (one
// block, or 2048/n whole blocks); each thread owns G groups of 8 consecutive
// coordinates.  The thread reads a group with one 16-byte load (and its signs
// with one 8-byte load) and applies the stages of index bits 0..2 in
// registers.  The stages of bits 3.. run in passes through LDS of up to four
// bits each: a thread gathers the coordinates that differ only in the pass's
// bits, applies their stages and scatters them back.  A last pass reads every group back in
// order, scales it by n^(-1/2), rounds to binary16 and writes it with 16-byte
// stores.  The segment sits in LDS as f32 with 8 padding words per 64, which
// keeps the stride-8 gathers of the first LDS pass on 64 distinct banks; the
// later passes read consecutive words.  Coordinates in [K, Kpad) read as zero:
// they form whole blocks, so their outputs are the zero padding the GEMV
// expects.  The paper's rotation holds the whole activation in one thread
// block, which bounds its width by the per-block shared memory; blockwise,
// the largest block here (32768 coordinates, 144 KiB of LDS) is independent of
// the activation width.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <string>

#include "leech_internal.h"

namespace leech {
namespace {

constexpr int kRotMaxLog = 15;     // blocks of up to 32768 coordinates
constexpr int kMinSegLog = 11;     // a workgroup covers at least 2048 coordinates

typedef uint32_t u32x4r __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2r __attribute__((ext_vector_type(2)));
typedef float f32x4r __attribute__((ext_vector_type(4)));

__host__ __device__ constexpr int seg_log(int k) { return k > kMinSegLog ? k : kMinSegLog; }
__host__ __device__ constexpr int seg_threads(int k) {
  return (1 << seg_log(k)) / 8 > 1024 ? 1024 : (1 << seg_log(k)) / 8;
}
__host__ __device__ constexpr int lds_words(int k) {
  return (1 << seg_log(k)) + ((1 << seg_log(k)) >> 3);
}
__device__ __forceinline__ int pad(int i) { return i + ((i >> 6) << 3); }

// Butterflies over the index bits [0, B) of E = 2^B values held in registers.
template <int E>
__device__ __forceinline__ void butterflies(float* v) {
#pragma unroll
  for (int st = 1; st < E; st <<= 1)
#pragma unroll
    for (int t = 0; t < E; ++t)
      if (!(t & st)) {
        const float a = v[t], b = v[t | st];
        v[t] = a + b;
        v[t | st] = a - b;
      }
}

__device__ __forceinline__ float h2f(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// One LDS pass over the index bits [LO, LO + BITS) of the segment.
template <int LO, int BITS, int T, int S>
__device__ __forceinline__ void lds_pass(float* buf, int tid) {
  constexpr int E = 1 << BITS;
  constexpr int NG = S / E;                 // groups in the segment
  constexpr int P = (NG + T - 1) / T;       // groups per thread (the last may idle)
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int q = tid + p * T;
    if (NG % T != 0 && q >= NG) break;
    const int b0 = ((q >> LO) << (LO + BITS)) | (q & ((1 << LO) - 1));
    float v[E];
#pragma unroll
    for (int t = 0; t < E; ++t) v[t] = buf[pad(b0 + (t << LO))];
    butterflies<E>(v);
#pragma unroll
    for (int t = 0; t < E; ++t) buf[pad(b0 + (t << LO))] = v[t];
  }
}

// Passes over index bits [LO, K2): the fewest of at most 4 bits each, the
// bits spread evenly over them (k = 10: 4 + 3 rather than 3 + 3 + 1), each
// after a barrier.  Bits are taken in increasing order, as the stages are.
template <int LO, int K2, int T, int S>
__device__ __forceinline__ void lds_passes(float* buf, int tid) {
  if constexpr (LO < K2) {
    constexpr int left = K2 - LO;
    constexpr int passes = (left + 3) / 4;
    constexpr int BITS = (left + passes - 1) / passes;
    __syncthreads();
    lds_pass<LO, BITS, T, S>(buf, tid);
    lds_passes<LO + BITS, K2, T, S>(buf, tid);
  }
}

// flags: bit 0 = x and signs allow vector loads, bit 1 = outputs allow vector stores
template <int K2>
__global__ __launch_bounds__(seg_threads(K2)) void rotate_kernel(
    const uint16_t* __restrict__ x, const int8_t* __restrict__ signs, int64_t K, int64_t Kpad,
    float norm, int flags, uint16_t* __restrict__ out, float* __restrict__ out32) {
  constexpr int S = 1 << seg_log(K2);
  constexpr int T = seg_threads(K2);
  constexpr int G = S / 8 / T;
  constexpr int B0 = K2 < 3 ? K2 : 3;     // index bits handled in registers
  extern __shared__ __attribute__((aligned(16))) float buf[];
  const int tid = threadIdx.x;
  const int64_t seg = (int64_t)blockIdx.x * S;

  float v[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t e0 = seg + 8 * (int64_t)(tid + g * T);
    if ((flags & 1) && e0 + 8 <= K) {
      const u32x4r h = *reinterpret_cast<const u32x4r*>(x + e0);
      u32x2r sg = {0x01010101u, 0x01010101u};
      if (signs) sg = *reinterpret_cast<const u32x2r*>(signs + e0);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t bits = __builtin_bit_cast(uint32_t, h2f(h[t >> 1] >> (16 * (t & 1))));
        // bit 7 of the sign byte set means −1: it becomes the f32 sign bit
        const uint32_t neg = (sg[t >> 2] >> (8 * (t & 3)) << 24) & 0x80000000u;
        v[g][t] = __builtin_bit_cast(float, bits ^ neg);
      }
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        float a = 0.0f;
        if (e0 + t < K) {
          a = h2f(x[e0 + t]);
          if (signs && signs[e0 + t] < 0) a = -a;
        }
        v[g][t] = a;
      }
    }
    butterflies<1 << B0>(v[g]);
    if constexpr (B0 < 3) {     // blocks shorter than 8: the other groups of 2^B0
#pragma unroll
      for (int t = 1 << B0; t < 8; t += 1 << B0) butterflies<1 << B0>(v[g] + t);
    }
  }

  if constexpr (K2 > 3) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float* d = buf + pad(8 * (tid + g * T));
      *reinterpret_cast<f32x4r*>(d) = {v[g][0], v[g][1], v[g][2], v[g][3]};
      *reinterpret_cast<f32x4r*>(d + 4) = {v[g][4], v[g][5], v[g][6], v[g][7]};
    }
    lds_passes<3, K2, T, S>(buf, tid);
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* d = buf + pad(8 * (tid + g * T));
      const f32x4r a = *reinterpret_cast<const f32x4r*>(d);
      const f32x4r b = *reinterpret_cast<const f32x4r*>(d + 4);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        v[g][t] = a[t];
        v[g][t + 4] = b[t];
      }
    }
  }

#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int64_t e0 = seg + 8 * (int64_t)(tid + g * T);
    uint32_t hw[4];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      float r = v[g][t] * norm;
      // rounded to f32 here and to binary16 below: the empty asm keeps the
      // compiler from fusing the product and the narrowing into one
      // mixed-precision multiply that would round only once
      asm("" : "+v"(r));
      v[g][t] = r;
      const uint32_t h = __builtin_bit_cast(uint16_t, (_Float16)r);
      hw[t >> 1] = (t & 1) ? (hw[t >> 1] | h << 16) : h;
    }
    if ((flags & 2) && e0 + 8 <= Kpad) {
      *reinterpret_cast<u32x4r*>(out + e0) = {hw[0], hw[1], hw[2], hw[3]};
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (e0 + t < Kpad) out[e0 + t] = (uint16_t)(hw[t >> 1] >> (16 * (t & 1)));
    }
    if (out32) {
      if ((flags & 2) && e0 + 8 <= K) {
        *reinterpret_cast<f32x4r*>(out32 + e0) = {v[g][0], v[g][1], v[g][2], v[g][3]};
        *reinterpret_cast<f32x4r*>(out32 + e0 + 4) = {v[g][4], v[g][5], v[g][6], v[g][7]};
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (e0 + t < K) out32[e0 + t] = v[g][t];
      }
    }
  }
}

typedef void (*RotateFn)(const uint16_t*, const int8_t*, int64_t, int64_t, float, int, uint16_t*,
                         float*);

template <int K2>
struct RotTable {
  static void fill(RotateFn* f) {
    f[K2] = rotate_kernel<K2>;
    RotTable<K2 - 1>::fill(f);
  }
};
template <>
struct RotTable<-1> {
  static void fill(RotateFn*) {}
};

int rot_fail(const char* what, hipError_t e) {
  return set_error(LEECH_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace
}  // namespace leech

using namespace leech;

extern "C" int leech_rotate_x(int64_t K, int64_t Kpad, const uint16_t* d_x, const int8_t* d_signs,
                              uint16_t* d_xr, float* d_xr32, void* stream) {
  clear_error();
  if (!d_x || !d_xr) return set_error(LEECH_E_ARG, "NULL argument");
  if (K <= 0 || Kpad < K) return set_error(LEECH_E_SHAPE, "need 0 < K <= Kpad");
  const int64_t n = K & -K;
  int k = 0;
  while ((int64_t)1 << k < n) ++k;
  if (k > kRotMaxLog)
    return set_error(LEECH_E_SHAPE, "power-of-two factor of K above 32768 is not supported");
  if (((uintptr_t)d_x & 1) || ((uintptr_t)d_xr & 1) || ((uintptr_t)d_xr32 & 3))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  const int64_t S = (int64_t)1 << seg_log(k);
  const int64_t grid = (Kpad + S - 1) / S;
  if (grid > 0x7fffffff) return set_error(LEECH_E_SHAPE, "activation too long");
  RotateFn fns[kRotMaxLog + 1];
  RotTable<kRotMaxLog>::fill(fns);
  const int flags = (((uintptr_t)d_x & 15) == 0 && ((uintptr_t)d_signs & 7) == 0 ? 1 : 0) |
                    (((uintptr_t)d_xr & 15) == 0 && ((uintptr_t)d_xr32 & 15) == 0 ? 2 : 0);
  // 2^(-k/2): exact for even k, rounded to f32 for odd k
  const float norm = (float)(1.0 / std::sqrt((double)n));
  const size_t shmem = k > 3 ? (size_t)lds_words(k) * sizeof(float) : 0;
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)fns[k],
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return rot_fail("hipFuncSetAttribute", e);
  }
  hipLaunchKernelGGL(fns[k], dim3((unsigned)grid), dim3(seg_threads(k)), shmem,
                     (hipStream_t)stream, d_x, d_signs, K, Kpad, norm, flags, d_xr, d_xr32);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return rot_fail("rotate launch", e);
  return LEECH_OK;
}
