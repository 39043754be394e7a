// a3: stable counting sort of assignments by expert id (the expert sorter).
//
// Three passes over chunks of kChunk assignments:
//   1. perm_hist     per-chunk histograms, counted in LDS;
//   2. perm_scan     one wave per expert: its count and, per chunk, the
//                    chunk's first slot relative to the expert's offset;
//   3. perm_scatter  one workgroup of 16 waves per chunk forms the expert
//                    offsets (exclusive scan of the counts); wave w places
//                    the chunk's assignments [64 w, 64 w + 64). Lanes holding
//                    the same expert find each other with ballots over the
//                    id bits (a lane's rank among its lower-numbered peers);
//                    per-wave expert counts in LDS, prefixed over the waves,
//                    order the waves. Slot = expert offset + chunk base +
//                    earlier waves' count + rank, which keeps the sort stable
//                    with no serial pass. (More experts than fit the per-wave
//                    counts: one wave walks the chunk 64 at a time with a
//                    running per-expert cursor instead.)
// Small inputs (one chunk) run all three steps in one workgroup, spread over
// its 16 waves when the experts' per-wave counts fit LDS.
// Integer counting only, so the result is exact and run-to-run identical.
#include "moe_dev.h"
#include "moe_launch.h"

namespace moe {

constexpr int kChunk = 1024;

__global__ __launch_bounds__(256) void perm_hist(const int32_t* __restrict__ ids, int A, int NE,
                                                 int32_t* __restrict__ hist) {
  extern __shared__ int32_t sh[];
  for (int e = threadIdx.x; e < NE; e += blockDim.x) sh[e] = 0;
  __syncthreads();
  const int base = blockIdx.x * kChunk;
  const int end = min(A, base + kChunk);
  for (int a = base + threadIdx.x; a < end; a += blockDim.x) {
    const int e = ids[a];
    if ((unsigned)e < (unsigned)NE) atomicAdd(&sh[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < NE; e += blockDim.x) hist[(size_t)blockIdx.x * NE + e] = sh[e];
}

// One wave per expert: lane l takes a contiguous run of the chunks, sums
// its counts, a wave-wide exclusive scan gives the run's first slot (relative
// to the expert's offset), and the lane then writes each chunk's base over
// its count; the expert's total goes to counts[e].
__device__ __forceinline__ int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int o = __shfl_up(v, d, kWave);
    if (lane >= d) v += o;
  }
  return v;
}

__global__ __launch_bounds__(256) void perm_scan(int32_t* __restrict__ hist, int nchunks, int NE,
                                                 int32_t* __restrict__ counts) {
  const int e = (int)blockIdx.x * 4 + (int)threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (e >= NE) return;
  const int per = (nchunks + kWave - 1) / kWave;
  const int c0 = min(nchunks, lane * per), c1 = min(nchunks, c0 + per);
  int sum = 0;
  for (int c = c0; c < c1; ++c) sum += hist[(size_t)c * NE + e];
  const int incl = wave_inclusive_scan(sum, lane);
  int run = incl - sum;
  for (int c = c0; c < c1; ++c) {
    int32_t* p = hist + (size_t)c * NE + e;
    const int n = *p;
    *p = run;  // chunk-local base (relative to the expert's offset)
    run += n;
  }
  if (lane == kWave - 1) counts[e] = incl;
}

// Stable in-order placement of up to kChunk assignments by one wave, given the
// first output slot of every expert for this chunk in cursor[] (LDS).
__device__ __forceinline__ void scatter_chunk(const int32_t* __restrict__ ids, int base, int end,
                                              int NE, int nbits, int32_t* cursor,
                                              int32_t* __restrict__ sorted,
                                              int32_t* __restrict__ pos) {
  const int lane = threadIdx.x % kWave;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
  for (int g = base; g < end; g += kWave) {
    const int a = g + lane;
    int e = a < end ? ids[a] : -1;
    const bool ok = (unsigned)e < (unsigned)NE;
    uint64_t peers = __ballot(ok);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = ok && ((e >> b) & 1);
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    if (ok) {
      const int rank = __popcll(peers & lt);
      const int dest = cursor[e] + rank;
      sorted[dest] = a;
      pos[a] = dest;
      // the highest peer advances the cursor past the whole group
      if ((peers >> lane) == 1ull) cursor[e] = dest + 1;
    }
  }
}

// One wave per chunk. The expert offsets (exclusive scan of counts) are
// formed by every wave from the counts (block 0 also writes them out); the
// cursor of expert e starts at its offset plus this chunk's base.
__global__ __launch_bounds__(64) void perm_scatter(const int32_t* __restrict__ ids, int A, int NE,
                                                   int nbits, const int32_t* __restrict__ hist,
                                                   const int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ offsets,
                                                   int32_t* __restrict__ sorted,
                                                   int32_t* __restrict__ pos) {
  extern __shared__ int32_t cursor[];
  const int lane = threadIdx.x;
  int carry = 0;
  for (int base = 0; base < NE; base += kWave) {
    const int e = base + lane;
    const int c = e < NE ? counts[e] : 0;
    const int incl = wave_inclusive_scan(c, lane);
    const int off = carry + incl - c;
    if (e < NE) {
      cursor[e] = off + hist[(size_t)blockIdx.x * NE + e];
      if (blockIdx.x == 0) offsets[e] = off;
    }
    carry += __shfl(incl, kWave - 1, kWave);
  }
  if (blockIdx.x == 0 && lane == 0) offsets[NE] = carry;
  __syncthreads();
  const int base = blockIdx.x * kChunk;
  scatter_chunk(ids, base, min(A, base + kChunk), NE, nbits, cursor, sorted, pos);
}

// Wave-level part of the 16-wave placement: assignment a of this lane (a < A
// taken), its expert e (ok: a valid id) and its rank among the wave's
// earlier lanes with the same expert; the group's highest lane records the
// group size in cnt[w * NE + e] (cnt zeroed beforehand, a barrier after).
__device__ __forceinline__ void wave_rank16(const int32_t* __restrict__ ids, int a, int A, int NE,
                                            int nbits, int32_t* cnt, int* e_out, bool* ok_out,
                                            int* rank_out) {
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int e = a < A ? ids[a] : -1;
  const bool ok = (unsigned)e < (unsigned)NE;
  uint64_t peers = __ballot(ok);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = ok && ((e >> b) & 1);
    const uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
  const int rank = __popcll(peers & lt);
  __syncthreads();  // cnt was zeroed by other threads
  if (ok && (peers >> lane) == 1ull) cnt[w * NE + e] = rank + 1;
  *e_out = e;
  *ok_out = ok;
  *rank_out = rank;
}

// Exclusive prefix of the 16 per-wave counts of expert threadIdx.x (in
// place); returns the expert's total. Call after a barrier.
__device__ __forceinline__ int prefix_waves16(int32_t* cnt, int NE) {
  int c = 0;
  if ((int)threadIdx.x < NE) {
    for (int v = 0; v < 16; ++v) {
      const int n = cnt[v * NE + threadIdx.x];
      cnt[v * NE + threadIdx.x] = c;
      c += n;
    }
  }
  return c;
}

// The scatter with 16 waves per chunk (NE <= kSmallNE).
__global__ __launch_bounds__(1024) void perm_scatter16(const int32_t* __restrict__ ids, int A,
                                                       int NE, int nbits,
                                                       const int32_t* __restrict__ hist,
                                                       const int32_t* __restrict__ counts,
                                                       int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ sorted,
                                                       int32_t* __restrict__ pos) {
  extern __shared__ int32_t sh[];
  int32_t* cnt = sh;            // [16][NE]
  int32_t* base = sh + 16 * NE;  // [NE]: expert offset + this chunk's base
  for (int i = threadIdx.x; i < 16 * NE; i += blockDim.x) cnt[i] = 0;
  const int c = (int)threadIdx.x < NE ? counts[threadIdx.x] : 0;
  int total;
  const int off = block_exclusive_scan_1024(c, &total);
  if ((int)threadIdx.x < NE) {
    base[threadIdx.x] = off + hist[(size_t)blockIdx.x * NE + threadIdx.x];
    if (blockIdx.x == 0) offsets[threadIdx.x] = off;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) offsets[NE] = total;
  const int a = (int)blockIdx.x * kChunk + (int)threadIdx.x;
  int e, rank;
  bool ok;
  wave_rank16(ids, a, A, NE, nbits, cnt, &e, &ok, &rank);
  __syncthreads();
  prefix_waves16(cnt, NE);
  __syncthreads();
  if (ok) {
    const int dest = base[e] + cnt[(threadIdx.x / kWave) * NE + e] + rank;
    sorted[dest] = a;
    pos[a] = dest;
  }
}

// All three steps in one workgroup of 1024 threads (A <= kChunk).
__global__ __launch_bounds__(1024) void perm_small(const int32_t* __restrict__ ids, int A, int NE,
                                                   int nbits, int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ offsets,
                                                   int32_t* __restrict__ sorted,
                                                   int32_t* __restrict__ pos) {
  extern __shared__ int32_t cursor[];
  for (int e = threadIdx.x; e < NE; e += blockDim.x) cursor[e] = 0;
  __syncthreads();
  for (int a = threadIdx.x; a < A; a += blockDim.x) {
    const int e = ids[a];
    if ((unsigned)e < (unsigned)NE) atomicAdd(&cursor[e], 1);
  }
  __syncthreads();
  int c0 = threadIdx.x < NE ? cursor[threadIdx.x] : 0;
  int c1 = threadIdx.x + 1024 < NE ? cursor[threadIdx.x + 1024] : 0;
  int total0, total1;
  const int p0 = block_exclusive_scan_1024(c0, &total0);
  const int p1 = block_exclusive_scan_1024(c1, &total1) + total0;
  if (threadIdx.x < NE) {
    counts[threadIdx.x] = c0;
    offsets[threadIdx.x] = p0;
    cursor[threadIdx.x] = p0;
  }
  if (threadIdx.x + 1024 < NE) {
    counts[threadIdx.x + 1024] = c1;
    offsets[threadIdx.x + 1024] = p1;
    cursor[threadIdx.x + 1024] = p1;
  }
  if (threadIdx.x == 0) offsets[NE] = total0 + total1;
  __syncthreads();
  if (threadIdx.x < kWave) scatter_chunk(ids, 0, A, NE, nbits, cursor, sorted, pos);
}

// Small inputs (A <= 1024, NE <= kSmallNE) in one workgroup where wave w
// places assignments [64 w, 64 w + 64): ballot ranks inside the wave, the
// per-wave count of every expert in LDS, and their exclusive prefix over the
// waves give each assignment its slot with no serial pass (stable: wave w's
// assignments precede wave w + 1's, lanes in order).
constexpr int kSmallNE = 512;

__global__ __launch_bounds__(1024) void perm_small16(const int32_t* __restrict__ ids, int A, int NE,
                                                     int nbits, int32_t* __restrict__ counts,
                                                     int32_t* __restrict__ offsets,
                                                     int32_t* __restrict__ sorted,
                                                     int32_t* __restrict__ pos) {
  extern __shared__ int32_t sh[];
  int32_t* cnt = sh;             // [16][NE]: per-wave counts, then their prefix over waves
  int32_t* off = sh + 16 * NE;   // [NE]: expert offsets
  for (int i = threadIdx.x; i < 16 * NE; i += blockDim.x) cnt[i] = 0;
  int e, rank;
  bool ok;
  wave_rank16(ids, (int)threadIdx.x, A, NE, nbits, cnt, &e, &ok, &rank);
  __syncthreads();
  const int c = prefix_waves16(cnt, NE);
  int total;
  const int p0 = block_exclusive_scan_1024(c, &total);
  if ((int)threadIdx.x < NE) {
    counts[threadIdx.x] = c;
    offsets[threadIdx.x] = p0;
    off[threadIdx.x] = p0;
  }
  if (threadIdx.x == 0) offsets[NE] = total;
  __syncthreads();
  if (ok) {
    const int dest = off[e] + cnt[(threadIdx.x / kWave) * NE + e] + rank;
    sorted[dest] = threadIdx.x;
    pos[threadIdx.x] = dest;
  }
}

size_t permute_workspace_bytes(int T, int NE, int k_total) {
  const long A = (long)T * k_total;
  const long nchunks = (A + kChunk - 1) / kChunk;
  return (size_t)((nchunks * NE * sizeof(int32_t) + 255) / 256 * 256);
}

hipError_t launch_permute(const int32_t* ids, int T, int NE, int k_total, int32_t* counts,
                          int32_t* offsets, int32_t* sorted, int32_t* pos, void* ws,
                          hipStream_t s) {
  const int A = T * k_total;
  int nbits = 0;
  while ((1 << nbits) < NE) ++nbits;
  const size_t lds = (size_t)NE * sizeof(int32_t);
  if (A <= kChunk && NE <= kSmallNE) {
    hipLaunchKernelGGL(perm_small16, dim3(1), dim3(1024), 17 * lds, s, ids, A, NE, nbits, counts,
                       offsets, sorted, pos);
    return hipGetLastError();
  }
  if (A <= kChunk) {
    hipLaunchKernelGGL(perm_small, dim3(1), dim3(1024), lds, s, ids, A, NE, nbits, counts, offsets,
                       sorted, pos);
    return hipGetLastError();
  }
  const int nchunks = (A + kChunk - 1) / kChunk;
  int32_t* hist = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(perm_hist, dim3(nchunks), dim3(256), lds, s, ids, A, NE, hist);
  hipLaunchKernelGGL(perm_scan, dim3((NE + 3) / 4), dim3(256), 0, s, hist, nchunks, NE, counts);
  if (NE <= kSmallNE)
    hipLaunchKernelGGL(perm_scatter16, dim3(nchunks), dim3(1024), 17 * lds, s, ids, A, NE, nbits,
                       hist, counts, offsets, sorted, pos);
  else
    hipLaunchKernelGGL(perm_scatter, dim3(nchunks), dim3(64), lds, s, ids, A, NE, nbits, hist,
                       counts, offsets, sorted, pos);
  return hipGetLastError();
}

}  // namespace moe
