// Load-time transcoder on gfx950 (§2.2 "Unfolding at load time": the 47-bit
// index is never decoded in the matvec; each block is expanded once, at load
// time, into its decoded-field record).  Format-v1 block codes -> the Planes14
// main stream, byte for byte what the host expansion writes.
//
// Geometry.  A thread owns 8 consecutive records of the stream (112 bytes,
// seven aligned 16-byte stores), so a wavefront writes 7 KiB contiguously.  For
// each record it maps the storage slot back to its (row, column block) in the
// wave-tile order, reads that block's 8-byte code (rows of a unit are nb
// blocks apart, so these reads gather) and decodes it with the shared
// format-v1 routines: a binary search over the class offsets, two or three
// 64-bit divisions into the mixed-radix digits, colex unranking of each
// level's positions straight into the three level-code planes, and the
// record's pair words built from them.  Each workgroup first copies the
// whole index table (60 KiB) into LDS, so the class search, the binomials and
// the codeword lists are LDS reads.  A grid-stride loop bounds the grid; every
// thread leaves once its slots pass the end of the stream.

#include <hip/hip_runtime.h>

#include <string>

#include "index_core.h"
#include "leech_internal.h"

namespace leech {
namespace {

constexpr int kTcThreads = 512;
static_assert(sizeof(IdxTable) % 16 == 0, "the table is copied to LDS in 16-byte words");
constexpr int kTcBlocksPerCu = 2;     // two workgroups (each with its LDS table copy) per CU
constexpr int kRecsPerThread = 8;
constexpr int kBytesPerThread = kRecsPerThread * kPlanes14Bytes;   // 112 = 7 × 16

typedef uint32_t u32x4t __attribute__((ext_vector_type(4)));

struct TranscodeArgs {
  const IdxTable* T;
  const uint64_t* code;
  uint8_t* main;
  uint32_t* bad;
  int64_t M, nb, n, tile_blocks, groups;
  uint64_t main_bytes;
  int C, R;
};

// Record words of one block: its three pair words and the 16-bit
// class | gain << 9 (the record's last two bytes).  Zeros for slots
// past the matrix and for codes that are not format-v1 codes.
__device__ __forceinline__ void record_words(const TranscodeArgs& a, const IdxTable& T, int64_t s,
                                             uint32_t w[4]) {
  w[0] = w[1] = w[2] = w[3] = 0;
  if (s >= a.n) return;
  const int64_t t = s / a.tile_blocks;
  const int64_t o = s - t * a.tile_blocks;
  const int64_t rows = min((int64_t)a.R, a.M - t * a.R);
  const int64_t g = o / (rows * a.C);
  const int64_t u = o - g * rows * a.C;
  const int64_t cols = min((int64_t)a.C, a.nb - g * a.C);
  const int64_t r = t * a.R + u / cols;
  const int64_t j = g * a.C + u % cols;
  uint16_t cls;
  uint8_t gain;
  uint32_t smask, p[3];
  if (!idx_decode(T, a.code[r * a.nb + j], &cls, &gain, &smask, p)) {
    atomicAdd(a.bad, 1u);
    return;
  }
  uint8_t code[kDim];
#pragma unroll
  for (int i = 0; i < kDim; ++i)
    code[i] = (uint8_t)((p[0] >> i & 1u) | (p[1] >> i & 1u) << 1 | (p[2] >> i & 1u) << 2);
  planes14_words(code, ~smask & 0xFFFFFFu, w);
  w[3] = (uint32_t)cls | (uint32_t)gain << 9;
}

__global__ __launch_bounds__(kTcThreads) void transcode_planes14_kernel(TranscodeArgs a) {
  // the index table (60.7 KB) in LDS: the class search, the binomials of the
  // colex unranking and the codeword lists are then LDS reads, not a chain of
  // dependent L2 reads per block
  __shared__ __attribute__((aligned(16))) IdxTable tab;
  {
    const u32x4t* src = reinterpret_cast<const u32x4t*>(a.T);
    u32x4t* dst = reinterpret_cast<u32x4t*>(&tab);
    for (int i = threadIdx.x; i < (int)(sizeof(IdxTable) / 16); i += kTcThreads) dst[i] = src[i];
  }
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * kTcThreads;
  for (int64_t t = (int64_t)blockIdx.x * kTcThreads + threadIdx.x;
       (uint64_t)t * kBytesPerThread < a.main_bytes; t += stride) {
    uint32_t out[28];
#pragma unroll
    for (int i = 0; i < kRecsPerThread; i += 2) {
      uint32_t x[4], y[4];
      record_words(a, tab, t * kRecsPerThread + i, x);
      record_words(a, tab, t * kRecsPerThread + i + 1, y);
      // two 14-byte records = seven words: the second starts at byte 14
      const int b = i / 2 * 7;
      out[b + 0] = x[0];
      out[b + 1] = x[1];
      out[b + 2] = x[2];
      out[b + 3] = (x[3] & 0xFFFFu) | y[0] << 16;
      out[b + 4] = y[0] >> 16 | y[1] << 16;
      out[b + 5] = y[1] >> 16 | y[2] << 16;
      out[b + 6] = y[2] >> 16 | y[3] << 16;
    }
    const uint64_t base = (uint64_t)t * kBytesPerThread;
#pragma unroll
    for (int q = 0; q < 7; ++q) {
      const uint64_t at = base + 16 * q;
      if (at + 16 <= a.main_bytes) {
        *reinterpret_cast<u32x4t*>(a.main + at) =
            u32x4t{out[4 * q], out[4 * q + 1], out[4 * q + 2], out[4 * q + 3]};
      } else {
        for (int e = 0; e < 16 && at + e < a.main_bytes; ++e)
          a.main[at + e] = (uint8_t)(out[4 * q + e / 4] >> (8 * (e % 4)));
      }
    }
  }
}

__global__ void clear_u32_kernel(uint32_t* p) { *p = 0; }

int tc_fail(const char* what, hipError_t e) {
  return set_error(LEECH_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace
}  // namespace leech

using namespace leech;

extern "C" int leech_transcode_planes14(const leech_layout_desc* desc, const void* d_index_table,
                                        const uint64_t* d_code, void* d_main, uint32_t* d_bad,
                                        void* stream) {
  clear_error();
  if (!desc || !d_index_table || !d_code || !d_main || !d_bad)
    return set_error(LEECH_E_ARG, "NULL argument");
  if (desc->layout != LEECH_PLANES14)
    return set_error(LEECH_E_LAYOUT, "the transcoder writes the Planes14 layout only");
  if (desc->M <= 0 || desc->Kpad <= 0 || desc->Kpad % kDim || desc->nb != desc->Kpad / kDim ||
      !geometry_ok(desc->lane_cols, desc->tile_rows))
    return set_error(LEECH_E_SHAPE, "descriptor shape is not valid");
  const int64_t n = desc->M * desc->nb;
  if (desc->main_bytes != (uint64_t)n * kPlanes14Bytes + kPadBytes)
    return set_error(LEECH_E_SHAPE, "descriptor size is not the Planes14 size of its shape");
  if (((uintptr_t)d_main & 15) || ((uintptr_t)d_code & 7) || ((uintptr_t)d_index_table & 15))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  Geometry geo(desc->M, desc->nb, desc->lane_cols, desc->tile_rows);
  TranscodeArgs a;
  a.T = (const IdxTable*)d_index_table;
  a.code = d_code;
  a.main = (uint8_t*)d_main;
  a.bad = d_bad;
  a.M = desc->M;
  a.nb = desc->nb;
  a.n = n;
  a.tile_blocks = (int64_t)geo.R * geo.nb;
  a.groups = geo.groups;
  a.main_bytes = desc->main_bytes;
  a.C = geo.C;
  a.R = geo.R;
  const uint64_t threads = (desc->main_bytes + kBytesPerThread - 1) / kBytesPerThread;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const uint64_t blocks = std::min<uint64_t>((threads + kTcThreads - 1) / kTcThreads,
                                             (uint64_t)kTcBlocksPerCu * (uint64_t)std::max(cus, 1));
  hipLaunchKernelGGL(clear_u32_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream, d_bad);
  hipLaunchKernelGGL(transcode_planes14_kernel, dim3((unsigned)blocks), dim3(kTcThreads), 0,
                     (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return tc_fail("transcode launch", e);
  return LEECH_OK;
}
