// Device half of libleech: fused Λ24(12) dequantize + GEMV for gfx950, its
// verification decode, the FP16 GEMV control and the no-weights control.
//
// Paper: §2.3 "The kernel" (a divergence-free read of decoded-field records
// with shifts, masks and a class-table lookup, f32 accumulation, a wavefront
// reduction), §3.2 (the four layouts), §3.3 (the no-weights control).
//
// Geometry (MI355X-specific; the paper's one-warp-per-row geometry is not
// used).  A workgroup owns one tile of tile_rows = 64 / lane_cols rows and
// walks its units: a unit is the ≤ 64 blocks of the tile's rows in lane_cols
// consecutive block columns, stored contiguously, so one wavefront step loads
// one unit with fully coalesced 128-byte lines (896 bytes of Planes14 records
// and 128 bytes of fp16 scales per step).  Lane (r, c) of a step handles block
// (tile·R + r, g·C + c) and accumulates its row's partial sum in a register;
// the activation x (binary16) and the class table are staged in LDS once per
// workgroup.  At the end the C lanes of a row are summed by an xor butterfly
// and the waves of the workgroup through LDS, in a fixed order, so the result
// depends only on (M, Kpad, lane_cols) and not on the layout.
//
// Every block is decoded to 12 packed binary16 pairs of its signed integer
// coordinates z_i (|z_i| ≤ 13, exact in binary16) and multiplied with x by
// v_dot2_f32_f16 (exact products, f32 sums); the block's factor
// scale · centroid[gain] / (4√m) is applied once per block (§2.3: one
// multiply per block).

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <string>

#include "leech_internal.h"

namespace leech {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4a __attribute__((ext_vector_type(4)));

constexpr int kNoWeights = 99;   // layout id of the no-weights control

struct GemvArgs {
  const uint8_t* main;
  const uint8_t* side0;
  const uint8_t* side1;
  const DevClass* table;        // global copy of LEECH_TABLE_DEVICE
  const uint32_t* codewords;    // Golay70 only
  const uint16_t* scale;        // fp16, storage order
  const uint16_t* x;            // fp16 [Kpad]
  float* y;                     // f32 [M]
  float cen0, cen1;
  int64_t M, nb, groups;
  int C, R, waves;
};

__device__ __forceinline__ uint32_t align(uint32_t hi, uint32_t lo, uint32_t s) {
  return __builtin_amdgcn_alignbit(hi, lo, s);
}

__device__ __forceinline__ half2_t pack2(int a, int b) {
  return __builtin_bit_cast(half2_t, __builtin_amdgcn_cvt_pkrtz((float)a, (float)b));
}

// Reinterpret a 32-bit word as two binary16 values.  Takes the word by value:
// applying __builtin_bit_cast directly to an ext_vector element (w.y) reads
// element 0 with this compiler, so vector elements go through this function.
__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// ---------------------------------------------------------------- decoders
// Each decoder fills z[24] (signed integer coordinates), cls and gain.

// Magnitude of level code c in class record t (codes 0..7).
__device__ __forceinline__ int mag_of(const DevClass& t, uint32_t lo, uint32_t hi, int code) {
  return (int)(__builtin_amdgcn_perm(hi, lo, (uint32_t)code) & 0xFFu);
}

// Planes14 record at byte offset off of base: class [0,9) | gain 9 |
// sign mask [10,34) | p0 [34,58) | p1 [58,82) | p2 [82,106).  The record
// starts at 14·b ≡ 0 or 2 (mod 4): a four-word window read with a 0- or
// 16-bit funnel shift (§2.3).
__device__ __forceinline__ void decode_planes14(const uint8_t* base, uint64_t off,
                                                const DevClass* tab, int* z, uint32_t& cls,
                                                uint32_t& gain) {
  u32x4 w = *(const u32x4*)(base + (off & ~3ull));
  uint32_t sh = (uint32_t)(off & 2) * 8u;
  uint32_t r0 = align(w.y, w.x, sh), r1 = align(w.z, w.y, sh), r2 = align(w.w, w.z, sh);
  uint32_t r3 = w.w >> sh;
  cls = r0 & 511u;
  gain = (r0 >> 9) & 1u;
  uint32_t sm = align(r1, r0, 10) & 0xFFFFFFu;
  uint32_t p0 = (r1 >> 2) & 0xFFFFFFu;
  uint32_t p1 = align(r2, r1, 26) & 0xFFFFFFu;
  uint32_t p2 = align(r3, r2, 18) & 0xFFFFFFu;
  const uint32_t* mw = (const uint32_t*)tab[cls].mag;
  uint32_t lo = mw[0], hi = mw[1];
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    int code = (int)((p0 >> i) & 1u) | (int)((p1 >> i) & 1u) << 1 | (int)((p2 >> i) & 1u) << 2;
    int a = mag_of(tab[cls], lo, hi, code);
    z[i] = ((sm >> i) & 1u) ? -a : a;
  }
}

// Planes12x: 12-byte record class | gain | sign mask | p0 | p1 | exception
// field [82,96); a nonzero field points into the tile's exception list of
// exact Planes14 records (§3.2).
__device__ __forceinline__ void decode_planes12x(const GemvArgs& a, uint64_t idx, int64_t tile,
                                                 const DevClass* tab, int* z, uint32_t& cls,
                                                 uint32_t& gain) {
  u32x3 w = *(const u32x3*)(a.main + idx * kPlanes12Bytes);
  uint32_t field = w.z >> kP12ExcShift;
  if (field) {
    uint32_t tb = ((const uint32_t*)a.side1)[tile];
    decode_planes14(a.side0, (uint64_t)(tb + field - 1) * kPlanes14Bytes, tab, z, cls, gain);
    return;
  }
  cls = w.x & 511u;
  gain = (w.x >> 9) & 1u;
  uint32_t sm = align(w.y, w.x, 10) & 0xFFFFFFu;
  uint32_t p0 = (w.y >> 2) & 0xFFFFFFu;
  uint32_t p1 = align(w.z, w.y, 26) & 0xFFFFFFu;
  const uint32_t* mw = (const uint32_t*)tab[cls].mag;
  uint32_t lo = mw[0], hi = mw[1];
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    int code = (int)((p0 >> i) & 1u) | (int)((p1 >> i) & 1u) << 1;
    int m = mag_of(tab[cls], lo, hi, code);
    z[i] = ((sm >> i) & 1u) ? -m : m;
  }
}

// Slot32: 16- or 20-byte records located through the unit's side entry (u64
// bitmap of 20-byte records, u32 word offset of the unit's first record); a
// fixed five-word window; one-hot masks of levels 1..L−1 at [34 + 24(k−1), …).
__device__ __forceinline__ void decode_slot32(const GemvArgs& a, int64_t unit, int lane,
                                              const DevClass* tab, int* z, uint32_t& cls,
                                              uint32_t& gain) {
  const uint8_t* ent = a.side0 + unit * kUnitEntryBytes;
  uint64_t bits = *(const uint64_t*)ent;
  uint32_t base = *(const uint32_t*)(ent + 8);
  uint32_t nbelow = (uint32_t)__builtin_popcountll(bits & ((1ull << lane) - 1ull));
  const uint32_t* rec = (const uint32_t*)(a.main + (uint64_t)base * 4 +
                                          (uint64_t)lane * kSlot32Small +
                                          (uint64_t)nbelow * (kSlot32Large - kSlot32Small));
  uint32_t r0 = rec[0], r1 = rec[1], r2 = rec[2], r3 = rec[3], r4 = rec[4];
  cls = r0 & 511u;
  gain = (r0 >> 9) & 1u;
  uint32_t L = tab[cls].info & 0xFFu;
  uint32_t sm = align(r1, r0, 10) & 0xFFFFFFu;
  uint32_t m1 = L > 1 ? (r1 >> 2) & 0xFFFFFFu : 0u;
  uint32_t m2 = L > 2 ? align(r2, r1, 26) & 0xFFFFFFu : 0u;
  uint32_t m3 = L > 3 ? align(r3, r2, 18) & 0xFFFFFFu : 0u;
  uint32_t m4 = L > 4 ? align(r4, r3, 10) & 0xFFFFFFu : 0u;
  const uint32_t* mw = (const uint32_t*)tab[cls].mag;
  uint32_t lo = mw[0], hi = mw[1];
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    int code = (int)((m1 >> i) & 1u) + 2 * (int)((m2 >> i) & 1u) + 3 * (int)((m3 >> i) & 1u) +
               4 * (int)((m4 >> i) & 1u);
    int m = mag_of(tab[cls], lo, hi, code);
    z[i] = ((sm >> i) & 1u) ? -m : m;
  }
}

// Golay70: 9-byte record class | gain | 12-bit codeword rank | 24 two-bit
// codes at [22,70) | exception flag 70.  The side of coordinate i is bit i of
// the codeword; its value is the class's g70[side][code].  Exceptions are
// exact Planes14 records located through the unit's side entry.
__device__ __forceinline__ void decode_golay70(const GemvArgs& a, uint64_t idx, int64_t unit,
                                               int lane, const DevClass* tab,
                                               const uint32_t* cw, int* z, uint32_t& cls,
                                               uint32_t& gain) {
  uint64_t off = idx * kGolay70Bytes;
  u32x3 w = *(const u32x3*)(a.main + (off & ~3ull));
  uint32_t sh = (uint32_t)(off & 3) * 8u;
  uint32_t r0 = align(w.y, w.x, sh), r1 = align(w.z, w.y, sh), r2 = w.z >> sh;
  if ((r2 >> 6) & 1u) {
    const uint8_t* ent = a.side1 + unit * kUnitEntryBytes;
    uint64_t bits = *(const uint64_t*)ent;
    uint32_t base = *(const uint32_t*)(ent + 8);
    uint32_t nbelow = (uint32_t)__builtin_popcountll(bits & ((1ull << lane) - 1ull));
    decode_planes14(a.side0, (uint64_t)(base + nbelow) * kPlanes14Bytes, tab, z, cls, gain);
    return;
  }
  cls = r0 & 511u;
  gain = (r0 >> 9) & 1u;
  uint32_t word = cw[(r0 >> 10) & 0xFFFu];
  uint64_t codes = ((((uint64_t)r2 << 32) | r1) << 10) | (r0 >> 22);
  const int8_t* v = &tab[cls].g70[0][0];
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    int side = (int)((word >> i) & 1u);
    int code = (int)((codes >> (2 * i)) & 3u);
    z[i] = v[side * 4 + code];
  }
}

// Decode the block at storage index idx of unit (tile, g), lane `lane`.
template <int LAYOUT>
__device__ __forceinline__ void decode_block(const GemvArgs& a, uint64_t idx, int64_t tile,
                                             int64_t unit, int lane, const DevClass* tab,
                                             const uint32_t* cw, int* z, uint32_t& cls,
                                             uint32_t& gain) {
  if constexpr (LAYOUT == LEECH_PLANES14)
    decode_planes14(a.main, idx * kPlanes14Bytes, tab, z, cls, gain);
  else if constexpr (LAYOUT == LEECH_PLANES12X)
    decode_planes12x(a, idx, tile, tab, z, cls, gain);
  else if constexpr (LAYOUT == LEECH_SLOT32)
    decode_slot32(a, unit, lane, tab, z, cls, gain);
  else
    decode_golay70(a, idx, unit, lane, tab, cw, z, cls, gain);
}

// ------------------------------------------------------------------- GEMV
template <int LAYOUT>
__global__ __launch_bounds__(1024) void gemv_kernel(GemvArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int64_t Kpad = a.nb * kDim;
  uint16_t* xs = (uint16_t*)smem;                                  // Kpad halves
  const size_t xbytes = ((size_t)Kpad * 2 + 15) & ~(size_t)15;
  DevClass* ts = (DevClass*)(smem + xbytes);                        // 512 records
  const size_t tbytes = (LAYOUT == kNoWeights) ? 0 : LEECH_DEVICE_TABLE_BYTES;
  uint32_t* cws = (uint32_t*)(smem + xbytes + tbytes);               // Golay70: 4096 words
  const size_t cbytes = (LAYOUT == LEECH_GOLAY70) ? 4096 * 4 : 0;
  float* red = (float*)(smem + xbytes + tbytes + cbytes);          // waves × 64

  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  {  // stage x, the class table (and the codeword table) into LDS
    const u32x4a* src = (const u32x4a*)a.x;
    u32x4a* dst = (u32x4a*)xs;
    for (int64_t k = tid; k < Kpad / 8; k += nthr) dst[k] = src[k];
    if (LAYOUT != kNoWeights) {
      const u32x4a* ts_src = (const u32x4a*)a.table;
      for (int k = tid; k < LEECH_DEVICE_TABLE_BYTES / 16; k += nthr) ((u32x4a*)ts)[k] = ts_src[k];
    }
    if (LAYOUT == LEECH_GOLAY70) {
      const u32x4a* c_src = (const u32x4a*)a.codewords;
      for (int k = tid; k < 4096 / 4; k += nthr) ((u32x4a*)cws)[k] = c_src[k];
    }
  }
  __syncthreads();

  const int64_t tile = blockIdx.x;
  const int R = a.R, C = a.C;
  const int R_t = (int)min((int64_t)R, a.M - tile * R);
  const int wave = tid >> 6, lane = tid & 63;
  const int rl = lane / C, cl = lane % C;
  float acc = 0.0f;

  for (int64_t g = wave; g < a.groups; g += a.waves) {
    const int C_g = (int)min((int64_t)C, a.nb - g * C);
    if (rl < R_t && cl < C_g) {
      const int ul = rl * C_g + cl;                    // lane inside the unit
      const uint64_t idx = (uint64_t)(tile * R * a.nb + g * R_t * C + ul);
      const int64_t j = g * C + cl;
      int z[kDim];
      uint32_t cls = 0, gain = 0;
      float f;
      if constexpr (LAYOUT == kNoWeights) {
#pragma unroll
        for (int i = 0; i < kDim; ++i) z[i] = 1;
        f = 1.0f;
      } else {
        decode_block<LAYOUT>(a, idx, tile, tile * a.groups + g, ul, ts, cws, z, cls, gain);
        const float s = half_bits_to_float(a.scale[idx]);
        f = (s * (gain ? a.cen1 : a.cen0)) * ts[cls].inv_norm;
      }
      const half2_t* xp = (const half2_t*)(xs + 24 * j);
      float s0 = 0.0f;
#pragma unroll
      for (int k = 0; k < 12; ++k) s0 = __builtin_amdgcn_fdot2(pack2(z[2 * k], z[2 * k + 1]), xp[k], s0, false);
      acc = __builtin_fmaf(s0, f, acc);
    }
  }
  for (int off = 1; off < C; off <<= 1) acc += __shfl_xor(acc, off);
  if (cl == 0 && rl < R_t) red[wave * 64 + rl] = acc;
  __syncthreads();
  if (tid < R_t) {
    float y = 0.0f;
    for (int w = 0; w < a.waves; ++w) y += red[w * 64 + tid];
    a.y[tile * R + tid] = y;
  }
}

// --------------------------------------------------------- decode export
template <int LAYOUT>
__global__ __launch_bounds__(256) void decode_kernel(GemvArgs a, int8_t* zout, uint16_t* cout,
                                                     uint8_t* gout) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.M * a.nb) return;
  const int64_t r = b / a.nb, j = b % a.nb;
  const int64_t tile = r / a.R, g = j / a.C;
  const int rl = (int)(r % a.R), cl = (int)(j % a.C);
  const int R_t = (int)min((int64_t)a.R, a.M - tile * a.R);
  const int C_g = (int)min((int64_t)a.C, a.nb - g * a.C);
  const int ul = rl * C_g + cl;
  const uint64_t idx = (uint64_t)(tile * a.R * a.nb + g * R_t * a.C + ul);
  int z[kDim];
  uint32_t cls = 0, gain = 0;
  decode_block<LAYOUT>(a, idx, tile, tile * a.groups + g, ul, a.table, a.codewords, z, cls,
                       gain);
  if (zout) {
    uint32_t* zo = (uint32_t*)(zout + b * kDim);
#pragma unroll
    for (int q = 0; q < 6; ++q)
      zo[q] = (uint32_t)(uint8_t)z[4 * q] | (uint32_t)(uint8_t)z[4 * q + 1] << 8 |
              (uint32_t)(uint8_t)z[4 * q + 2] << 16 | (uint32_t)(uint8_t)z[4 * q + 3] << 24;
  }
  if (cout) cout[b] = (uint16_t)cls;
  if (gout) gout[b] = (uint8_t)gain;
}

// ------------------------------------------------------ FP16 GEMV control
// One wavefront per row; lanes stream 16-byte chunks of the row (1 KiB per
// wavefront load); x staged in LDS; f32 accumulation with v_dot2_f32_f16.
__global__ __launch_bounds__(512) void fp16_gemv_kernel(const uint16_t* __restrict__ W,
                                                        const uint16_t* __restrict__ x,
                                                        float* __restrict__ y, int64_t M,
                                                        int64_t K) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int64_t K8 = K / 8;
  u32x4a* xs = (u32x4a*)smem;
  for (int64_t k = threadIdx.x; k < K8; k += blockDim.x) xs[k] = ((const u32x4a*)x)[k];
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
  if (row >= M) return;
  const u32x4a* wr = (const u32x4a*)(W + row * K);
  float acc = 0.0f;
  for (int64_t c = lane; c < K8; c += 64) {
    u32x4a w = wr[c];
    u32x4a xv = xs[c];
    acc = __builtin_amdgcn_fdot2(as_h2(w.x), as_h2(xv.x), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.y), as_h2(xv.y), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.z), as_h2(xv.z), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.w), as_h2(xv.w), acc, false);
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) y[row] = acc;
}

// ------------------------------------------------------------- launching
static int hip_fail(const char* what, hipError_t e) {
  return set_error(LEECH_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

static int waves_for(int64_t groups) { return (int)std::max<int64_t>(1, std::min<int64_t>(8, groups)); }

static int check_desc_device(const leech_layout_desc* d) {
  if (!d) return set_error(LEECH_E_ARG, "desc is NULL");
  if (d->M <= 0 || d->Kpad <= 0 || d->Kpad % kDim || d->nb != d->Kpad / kDim)
    return set_error(LEECH_E_SHAPE, "descriptor shape is not valid");
  if (d->lane_cols != choose_lane_cols(d->M))
    return set_error(LEECH_E_SHAPE, "descriptor lane_cols does not match its M");
  return LEECH_OK;
}

static GemvArgs make_args(const leech_layout_desc* d) {
  GemvArgs a;
  std::memset(&a, 0, sizeof a);
  a.M = d->M;
  a.nb = d->nb;
  a.C = d->lane_cols;
  a.R = kWave / d->lane_cols;
  a.groups = (d->nb + a.C - 1) / a.C;
  a.waves = waves_for(a.groups);
  return a;
}

template <int LAYOUT>
static int launch_gemv(const GemvArgs& a, hipStream_t st) {
  size_t xbytes = ((size_t)a.nb * kDim * 2 + 15) & ~(size_t)15;
  size_t shmem = xbytes + (LAYOUT == kNoWeights ? 0 : LEECH_DEVICE_TABLE_BYTES) +
                 (LAYOUT == LEECH_GOLAY70 ? 4096 * 4 : 0) + (size_t)a.waves * 64 * 4;
  if (shmem > 160 * 1024)
    return set_error(LEECH_E_SHAPE, "Kpad too large for the LDS-staged activation");
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)gemv_kernel<LAYOUT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return hip_fail("hipFuncSetAttribute", e);
  }
  int64_t tiles = (a.M + a.R - 1) / a.R;
  hipLaunchKernelGGL(gemv_kernel<LAYOUT>, dim3((unsigned)tiles), dim3(64 * a.waves), shmem, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("gemv launch", e);
  return LEECH_OK;
}

template <int LAYOUT>
static int launch_decode(const GemvArgs& a, int8_t* z, uint16_t* c, uint8_t* g, hipStream_t st) {
  int64_t n = a.M * a.nb;
  hipLaunchKernelGGL(decode_kernel<LAYOUT>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     a, z, c, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("decode launch", e);
  return LEECH_OK;
}

}  // namespace leech

using namespace leech;

extern "C" {

int leech_gemv(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
               const void* d_side1, const void* d_class_table, const void* d_codewords,
               const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
               float* d_y, void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_main || !d_class_table || !d_scale || !centroid || !d_x || !d_y)
    return set_error(LEECH_E_ARG, "NULL argument");
  if ((desc->side_bytes[0] && !d_side0) || (desc->side_bytes[1] && !d_side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  if (desc->layout == LEECH_GOLAY70 && !d_codewords)
    return set_error(LEECH_E_ARG, "GOLAY70 needs the codeword table");
  if (((uintptr_t)d_x & 15) || ((uintptr_t)d_main & 3) || ((uintptr_t)d_class_table & 15) ||
      ((uintptr_t)d_codewords & 15) || ((uintptr_t)d_side0 & 3) || ((uintptr_t)d_side1 & 7))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.main = (const uint8_t*)d_main;
  a.side0 = (const uint8_t*)d_side0;
  a.side1 = (const uint8_t*)d_side1;
  a.table = (const DevClass*)d_class_table;
  a.codewords = (const uint32_t*)d_codewords;
  a.scale = d_scale;
  a.x = d_x;
  a.y = d_y;
  a.cen0 = centroid[0];
  a.cen1 = centroid[1];
  hipStream_t st = (hipStream_t)stream;
  switch (desc->layout) {
    case LEECH_SLOT32: return launch_gemv<LEECH_SLOT32>(a, st);
    case LEECH_PLANES14: return launch_gemv<LEECH_PLANES14>(a, st);
    case LEECH_PLANES12X: return launch_gemv<LEECH_PLANES12X>(a, st);
    case LEECH_GOLAY70: return launch_gemv<LEECH_GOLAY70>(a, st);
    default: return set_error(LEECH_E_LAYOUT, "unknown layout");
  }
}

int leech_decode_blocks(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                        const void* d_side1, const void* d_class_table,
                        const void* d_codewords, int8_t* d_z, uint16_t* d_class_id,
                        uint8_t* d_gain_bit, void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_main || !d_class_table) return set_error(LEECH_E_ARG, "NULL argument");
  if ((desc->side_bytes[0] && !d_side0) || (desc->side_bytes[1] && !d_side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  if (desc->layout == LEECH_GOLAY70 && !d_codewords)
    return set_error(LEECH_E_ARG, "GOLAY70 needs the codeword table");
  if (((uintptr_t)d_z & 3) || ((uintptr_t)d_main & 3) || ((uintptr_t)d_side1 & 7))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.main = (const uint8_t*)d_main;
  a.side0 = (const uint8_t*)d_side0;
  a.side1 = (const uint8_t*)d_side1;
  a.table = (const DevClass*)d_class_table;
  a.codewords = (const uint32_t*)d_codewords;
  hipStream_t st = (hipStream_t)stream;
  switch (desc->layout) {
    case LEECH_SLOT32: return launch_decode<LEECH_SLOT32>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_PLANES14: return launch_decode<LEECH_PLANES14>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_PLANES12X: return launch_decode<LEECH_PLANES12X>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_GOLAY70: return launch_decode<LEECH_GOLAY70>(a, d_z, d_class_id, d_gain_bit, st);
    default: return set_error(LEECH_E_LAYOUT, "unknown layout");
  }
}

int leech_fp16_gemv_ref(int64_t M, int64_t K, const uint16_t* d_W, const uint16_t* d_x,
                        float* d_y, void* stream) {
  clear_error();
  if (!d_W || !d_x || !d_y) return set_error(LEECH_E_ARG, "NULL argument");
  if (M <= 0 || K <= 0 || K % 8) return set_error(LEECH_E_SHAPE, "need M > 0, K > 0, K % 8 == 0");
  if (((uintptr_t)d_W & 15) || ((uintptr_t)d_x & 15))
    return set_error(LEECH_E_ARG, "W and x must be 16-byte aligned");
  size_t shmem = (size_t)K * 2;
  if (shmem > 160 * 1024) return set_error(LEECH_E_SHAPE, "K too large for the LDS-staged x");
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)fp16_gemv_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return hip_fail("hipFuncSetAttribute", e);
  }
  const int waves = 8;
  hipLaunchKernelGGL(fp16_gemv_kernel, dim3((unsigned)((M + waves - 1) / waves)), dim3(64 * waves),
                     shmem, (hipStream_t)stream, d_W, d_x, d_y, M, K);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("fp16 gemv launch", e);
  return LEECH_OK;
}

int leech_noweights_ctrl(const leech_layout_desc* desc, const uint16_t* d_x, float* d_y,
                         void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_x || !d_y) return set_error(LEECH_E_ARG, "NULL argument");
  if ((uintptr_t)d_x & 15) return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.x = d_x;
  a.y = d_y;
  return launch_gemv<kNoWeights>(a, (hipStream_t)stream);
}

}  // extern "C"
