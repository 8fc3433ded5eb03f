// Memory-system probe for the roofline of the gather-bound kernels (measurement only).
//
// k_probe_gather replays an index stream with the access pattern of the SpMM's
// neighbour gathers and nothing else: row idx[k] of a row-major table (row_bytes per
// row, read as LPN = row_bytes / 16 lanes of one 16-byte load each) is loaded for every
// k, kInflightProbe rows in flight per lane group, and summed.  A wavefront owns a
// contiguous range of kProbeChunk indices; its NPW = 64 / LPN lane groups take every
// NPW-th index, and one row of sums per wavefront is stored, so the stores are about
// 1/kProbeChunk of the gathered bytes.  Replaying the SpMM's own column-index stream
// over a table of p's size gives the time of its gathers alone; replaying other
// streams (folded into a small footprint, uniform over a large one) separates the
// rates of L2 hits, Infinity-Cache hits and DRAM reads.
//
// With S > 1 slices the table's rows are S * row_bytes wide and the grid is S times
// larger: block b gathers slice b % S (row_bytes at offset (b % S) * row_bytes of each
// row) for index chunk b / S.  Blocks are dispatched to the XCDs round-robin, so with S
// dividing 8 every XCD gathers one slice of the rows only, and each XCD's L2 caches a
// footprint S times smaller than the whole table.
#include <hip/hip_runtime.h>

#include "erc_common.h"

namespace erc {
namespace {

constexpr int kProbeChunk = 2048;
constexpr int kInflightProbe = 8;

template <int LPN>
__global__ __launch_bounds__(kBlock) void k_probe_gather(const int32_t* __restrict__ idx,
                                                         int64_t count,
                                                         const float4* __restrict__ table,
                                                         int64_t rows, int slices,
                                                         float4* __restrict__ out) {
  constexpr int NPW = 64 / LPN;
  const int lane = threadIdx.x & 63;
  const int grp = lane / LPN;
  const int sub = lane % LPN;
  const int slice = static_cast<int>(blockIdx.x % static_cast<unsigned>(slices));
  const int64_t unit = blockIdx.x / static_cast<unsigned>(slices);
  const int64_t wave = unit * kWavesPerBlock + (threadIdx.x >> 6);
  // row j's slice starts at float4 (j * slices + slice) * LPN
  const int64_t rstride = static_cast<int64_t>(slices) * LPN;
  table += static_cast<int64_t>(slice) * LPN;
  const int64_t b = wave * kProbeChunk;
  if (b >= count) return;
  const int64_t e = min(b + static_cast<int64_t>(kProbeChunk), count);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int64_t k0 = b + grp; k0 < e; k0 += static_cast<int64_t>(NPW) * kInflightProbe) {
    float4 v[kInflightProbe];
#pragma unroll
    for (int u = 0; u < kInflightProbe; ++u) {
      const int64_t k = k0 + static_cast<int64_t>(u) * NPW;
      int64_t j = 0;
      if (k < e) {
        j = idx[k];
        if (j < 0 || j >= rows) j = 0;  // out-of-range indices read row 0
      }
      v[u] = (k < e) ? table[j * rstride + sub] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < kInflightProbe; ++u) {
      acc.x += v[u].x;
      acc.y += v[u].y;
      acc.z += v[u].z;
      acc.w += v[u].w;
    }
  }
#pragma unroll
  for (int off = LPN; off < 64; off <<= 1) {
    acc.x += __shfl_xor(acc.x, off);
    acc.y += __shfl_xor(acc.y, off);
    acc.z += __shfl_xor(acc.z, off);
    acc.w += __shfl_xor(acc.w, off);
  }
  if (lane < LPN) out[(wave * slices + slice) * LPN + sub] = acc;
}

template <int LPN>
hipError_t probe_t(const int32_t* idx, int64_t count, const void* table, int64_t rows,
                   int slices, void* out, hipStream_t s) {
  // every wave's chunk starts below count, so each stores inside out's
  // probe_out_rows(count) * slices rows
  const int64_t waves = (count + kProbeChunk - 1) / kProbeChunk;
  const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL((k_probe_gather<LPN>), dim3(static_cast<unsigned>(blocks * slices)),
                     dim3(kBlock), 0, s, idx, count, static_cast<const float4*>(table), rows,
                     slices, static_cast<float4*>(out));
  return hipGetLastError();
}

}  // namespace

int64_t probe_out_rows(int64_t count) { return (count + kProbeChunk - 1) / kProbeChunk; }

hipError_t launch_probe_gather(const int32_t* idx, int64_t count, const void* table, int64_t rows,
                               int row_bytes, int slices, void* out, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (slices < 1 || slices > 64) return hipErrorInvalidValue;
  switch (row_bytes / 16) {
    case 4: return probe_t<4>(idx, count, table, rows, slices, out, s);
    case 8: return probe_t<8>(idx, count, table, rows, slices, out, s);
    case 16: return probe_t<16>(idx, count, table, rows, slices, out, s);
    case 32: return probe_t<32>(idx, count, table, rows, slices, out, s);
    case 64: return probe_t<64>(idx, count, table, rows, slices, out, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace erc
