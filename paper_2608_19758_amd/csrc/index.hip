// The selection as a CSR index of 64-token key tiles (Sec. 3.3 Eq. csr; the
// compaction of Algorithm 1, where logical blocks are expanded to B/64
// physical tiles). Segment s = (b * Hkv + h) * nbmax + I follows the mask rows; its
// entries are, ascending, the key tiles j (keys 64j .. 64j+63) of every kept
// block J: 2J, and 2J+1 when that tile starts before the sequence's last key.
//
// Three passes: counts per segment (one workgroup each), one exclusive scan
// over the segments in a single workgroup (contiguous segment ranges per
// thread), and the writes (one workgroup per segment, kept blocks ranked with
// wave ballots). Every entry but the last block's is a pair, so block J's
// first tile goes to offset + 2 * (kept blocks before J).
#include "kernels.h"

namespace fp2 {

namespace {

constexpr int kTile = 64;   // keys per physical tile

// Segment -> the last key block visible to its tile (that of its last row)
// and the KV length; false for a tile past its sequence.
__device__ __forceinline__ bool segment(const Problem& p, int s, int& Ia, int& Lk) {
  const int I = s % p.nbmax, bh = s / p.nbmax, b = bh / p.hkv;
  const int Lq = p.cu[b + 1] - p.cu[b];
  if (I * p.qtile >= Lq) return false;
  Lk = p.cuk[b + 1] - p.cuk[b];
  Ia = (Lk - Lq + min(Lq, (I + 1) * p.qtile) - 1) / kBlock;   // block of the tile's last row
  return true;
}

__device__ __forceinline__ int tiles_of(int J, int Lk) {
  return (2 * J + 1) * kTile < Lk ? 2 : 1;
}

__global__ __launch_bounds__(256) void csr_count_kernel(Problem p, const uint8_t* __restrict__ mask,
                                                        int32_t* __restrict__ counts) {
  __shared__ int red[4];
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int Ia = -1, Lk = 0;
  const bool live = segment(p, s, Ia, Lk);
  const uint8_t* mrow = mask + (int64_t)s * p.nbk;
  int n = 0;
  if (live)
    for (int J = tid; J <= Ia; J += 256) n += (mrow[J] & 1) ? tiles_of(J, Lk) : 0;
  for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o, 64);
  if (lane == 0) red[w] = n;
  __syncthreads();
  if (tid == 0) counts[s] = red[0] + red[1] + red[2] + red[3];
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void csr_scan_kernel(int nseg,
                                                                const int32_t* __restrict__ counts,
                                                                int32_t* __restrict__ offsets) {
  __shared__ int sh[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per = (nseg + kScanThreads - 1) / kScanThreads;
  const int s0 = min(nseg, tid * per), s1 = min(nseg, s0 + per);
  int sum = 0;
  for (int s = s0; s < s1; ++s) sum += counts[s];
  int inc = sum;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  int base = inc - sum;
  for (int k = 0; k < w; ++k) base += sh[k];
  for (int s = s0; s < s1; ++s) {
    offsets[s] = base;
    base += counts[s];
  }
  if (tid == kScanThreads - 1) offsets[nseg] = base;
}

__global__ __launch_bounds__(256) void csr_write_kernel(Problem p, const uint8_t* __restrict__ mask,
                                                        const int32_t* __restrict__ offsets,
                                                        int32_t* __restrict__ indices) {
  __shared__ int red[4];
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int Ia = -1, Lk = 0;
  if (!segment(p, s, Ia, Lk)) return;
  const uint8_t* mrow = mask + (int64_t)s * p.nbk;
  int32_t* out = indices + offsets[s];
  int base = 0;   // kept blocks before this chunk
  for (int J0 = 0; J0 <= Ia; J0 += 256) {
    const int J = J0 + tid;
    const bool keep = J <= Ia && (mrow[J] & 1);
    const uint64_t bal = __ballot(keep);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) red[w] = __popcll(bal);
    __syncthreads();
    int wpre = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      wpre += k < w ? red[k] : 0;
      tot += red[k];
    }
    if (keep) {
      const int at = 2 * (base + wpre + before);
      out[at] = 2 * J;
      if (tiles_of(J, Lk) == 2) out[at + 1] = 2 * J + 1;
    }
    base += tot;
  }
}

}  // namespace

hipError_t launch_mask_to_csr(const Problem& p, const uint8_t* mask, int32_t* counts,
                              int32_t* offsets, int32_t* indices, hipStream_t s) {
  const int nseg = p.batch * p.hkv * p.nbmax;
  if (nseg == 0) return hipSuccess;
  csr_count_kernel<<<nseg, 256, 0, s>>>(p, mask, counts);
  csr_scan_kernel<<<1, kScanThreads, 0, s>>>(nseg, counts, offsets);
  csr_write_kernel<<<nseg, 256, 0, s>>>(p, mask, offsets, indices);
  return hipGetLastError();
}

}  // namespace fp2
