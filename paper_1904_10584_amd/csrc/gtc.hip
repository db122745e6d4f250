// Gradient Threshold Compression: encode with residual error feedback and
// ordered compaction of the sent elements into (index << 1 | sign) words,
// and the matching decode.  Exact fp32 (single adds/subtracts, IEEE
// subnormals), so the result is bit-identical to the element-wise definition.
//
// Encode runs in two launches over tiles of 4096 elements:
//   1. update: a = r + g; r <- a -+ tau where |a| > tau; a 2-bit code per
//      element (sent, sign) is packed 16 codes per thread word; per-tile count.
//      Reads g and r, writes r: 12 bytes per element plus 1/4 byte of codes.
//   2. compact: each tile's block sums the counts of the tiles before it
//      (up to 8192 tiles; beyond, a one-block scan turns the counts into
//      offsets first), ranks its sent elements in index order into LDS and
//      writes their words contiguously.
// Measured alternatives (a single resident launch with the codes kept on
// chip, super-tile counts by atomics, a fused scan) streamed the update
// slower or serialised on atomics.
// Decode builds each 4096-element tile of the dense update in LDS (zero or
// the existing values, then +-tau at the indices of the tile's words, found
// by binary search in the ascending word list) and writes it once.  The
// aggregate of several workers' streams (below) counts signs per element in
// LDS integers and scales by tau once.
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int TILE = (int)GTC_TILE;  // elements per tile
constexpr int TPB = 256;          // threads per block; 16 elements each
// Element e of a tile is handled by thread (e % 1024) / 4 as item
// (e / 1024) * 4 + e % 4: four float4 groups at stride 1024.

template <bool ALIGNED>
__global__ __launch_bounds__(TPB) void gtc_update(int64_t n, const float* __restrict__ g,
                                                  float* __restrict__ r, float tau,
                                                  uint32_t* __restrict__ codes,
                                                  int32_t* __restrict__ tile_count) {
  __shared__ int wsum[TPB / 64];
  const int64_t base = (int64_t)blockIdx.x * TILE;
  uint32_t code = 0;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp) {
    const int64_t e = base + grp * 1024 + threadIdx.x * 4;
    float gv[4], rv[4];
    if (ALIGNED && e + 3 < n) {
      const float4 g4 = *reinterpret_cast<const float4*>(g + e);
      const float4 r4 = *reinterpret_cast<const float4*>(r + e);
      gv[0] = g4.x; gv[1] = g4.y; gv[2] = g4.z; gv[3] = g4.w;
      rv[0] = r4.x; rv[1] = r4.y; rv[2] = r4.z; rv[3] = r4.w;
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        gv[c] = e + c < n ? g[e + c] : 0.f;
        rv[c] = e + c < n ? r[e + c] : 0.f;
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float a = rv[c] + gv[c];
      uint32_t k = 0;
      float nr = a;
      if (a > tau) { nr = a - tau; k = 1u; }
      else if (a < -tau) { nr = a + tau; k = 3u; }
      rv[c] = nr;
      code |= k << (2 * (grp * 4 + c));
    }
    if (ALIGNED && e + 3 < n) {
      *reinterpret_cast<float4*>(r + e) = make_float4(rv[0], rv[1], rv[2], rv[3]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (e + c < n) r[e + c] = rv[c];
    }
  }
  codes[(int64_t)blockIdx.x * TPB + threadIdx.x] = code;
  int cnt = __popc(code & 0x55555555u);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) tile_count[blockIdx.x] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
}

// Exclusive prefix of tile counts (in place) and the total, one block.
__global__ __launch_bounds__(1024) void gtc_scan(int32_t* __restrict__ tile_count, int64_t ntiles,
                                                 int64_t* __restrict__ total) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (ntiles + 1023) / 1024;
  const int64_t lo = t * per, hi = lo + per < ntiles ? lo + per : ntiles;
  int64_t s = 0;
  for (int64_t i = lo; i < hi; ++i) s += tile_count[i];
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {  // Hillis-Steele inclusive scan
    int64_t v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int64_t run = part[t] - s;  // exclusive
  for (int64_t i = lo; i < hi; ++i) {
    const int32_t c = tile_count[i];
    tile_count[i] = (int32_t)run;
    run += c;
  }
  if (t == 1023) *total = part[1023];
}

// Ranks of one tile's sent elements, in index order: thread t's code word
// covers elements 1024 grp + 4 t + c of the tile (grp, c < 4), so per group
// the 16-bit field counts are scanned over the threads.  Each word goes to
// its place in the tile's LDS buffer; returns the tile's word count.
__device__ __forceinline__ uint32_t rank_tile(uint32_t code, uint32_t tile_base, uint32_t* buf,
                                              uint64_t* wtot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t mine = 0;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp)
    mine |= (uint64_t)__popc((code >> (8 * grp)) & 0x55u) << (16 * grp);
  uint64_t inc = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t v = __shfl_up(inc, o, 64);
    if (lane >= o) inc += v;
  }
  if (lane == 63) wtot[wave] = inc;
  __syncthreads();
  uint64_t before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < TPB / 64; ++w) {
    if (w < wave) before += wtot[w];
    total += wtot[w];
  }
  const uint64_t excl = before + inc - mine;
  const uint32_t e0 = tile_base + threadIdx.x * 4;
  uint32_t lp = 0;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp) {
    uint32_t p = lp + (uint32_t)((excl >> (16 * grp)) & 0xFFFFu);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t k = (code >> (2 * (grp * 4 + c))) & 3u;
      if (k & 1u) buf[p++] = ((e0 + grp * 1024 + c) << 1) | (k >> 1);
    }
    lp += (uint32_t)((total >> (16 * grp)) & 0xFFFFu);
  }
  __syncthreads();
  return lp;
}

// Compaction for up to OWN_PREFIX_TILES tiles: each block sums the counts of
// every earlier tile itself (16-byte loads, all issued at once; they hit the
// L2), so no scan launch sits between the update and the compaction.  The
// tile's words are ranked into LDS and leave as consecutive 4-byte stores.
// The last tile's block writes the total.
constexpr int64_t OWN_PREFIX_TILES = 8 * TPB * 4;  // 8192 tiles: n <= 2^25

__global__ __launch_bounds__(TPB) void gtc_compact_own_prefix(int64_t ntiles,
                                                              const uint32_t* __restrict__ codes,
                                                              const int32_t* __restrict__ tile_count,
                                                              uint32_t* __restrict__ words,
                                                              int64_t* __restrict__ total_out) {
  __shared__ uint32_t buf[TILE];
  __shared__ uint64_t wtot[TPB / 64];
  __shared__ uint32_t wpre[TPB / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t t = blockIdx.x;
  const uint32_t code = codes[t * TPB + threadIdx.x];
  uint32_t pre = 0;
  {
    int4 q[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t j = ((int64_t)i * TPB + threadIdx.x) * 4;
      if (j + 3 < t) {
        q[i] = *reinterpret_cast<const int4*>(tile_count + j);
      } else {
        q[i].x = j < t ? tile_count[j] : 0;
        q[i].y = j + 1 < t ? tile_count[j + 1] : 0;
        q[i].z = j + 2 < t ? tile_count[j + 2] : 0;
        q[i].w = 0;
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) pre += (uint32_t)((q[i].x + q[i].y) + (q[i].z + q[i].w));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) pre += __shfl_xor(pre, o, 64);
  if (lane == 0) wpre[wave] = pre;
  const uint32_t lp = rank_tile(code, (uint32_t)(t * TILE), buf, wtot);  // (its barrier orders wpre)
  const uint32_t pos = ((wpre[0] + wpre[1]) + wpre[2]) + wpre[3];
  for (uint32_t i = threadIdx.x; i < lp; i += TPB) words[pos + i] = buf[i];
  if (t == ntiles - 1 && threadIdx.x == 0) *total_out = (int64_t)pos + lp;
}

// Compaction after a scan of the tile counts into offsets (more tiles).
__global__ __launch_bounds__(TPB) void gtc_compact(const uint32_t* __restrict__ codes,
                                                   const int32_t* __restrict__ tile_off,
                                                   uint32_t* __restrict__ words) {
  __shared__ uint32_t buf[TILE];
  __shared__ uint64_t wtot[TPB / 64];
  const int64_t t = blockIdx.x;
  const uint32_t code = codes[t * TPB + threadIdx.x];
  const uint32_t pos = (uint32_t)tile_off[t];
  const uint32_t lp = rank_tile(code, (uint32_t)(t * TILE), buf, wtot);
  for (uint32_t i = threadIdx.x; i < lp; i += TPB) words[pos + i] = buf[i];
}

__device__ __forceinline__ int64_t lower_bound_words(const uint32_t* w, int64_t cnt, uint32_t key) {
  int64_t lo = 0, hi = cnt;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (w[mid] < key) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// The same, found by a whole wave: each round the 64 lanes probe 64 evenly
// spaced positions of the remaining range [lo, hi] and a ballot of
// (word < key), true on a prefix of the lanes, narrows it about 65-fold; the
// last 64 or fewer candidates are tested at once.  About five rounds of
// dependent loads for 2^24 words instead of 24.  Wave-uniform result.
__device__ __forceinline__ int64_t lower_bound_wave(const uint32_t* w, int64_t cnt, uint32_t key,
                                                    int lane) {
  int64_t lo = 0, hi = cnt;  // the first word >= key lies in [lo, hi] (hi: none)
  while (hi - lo > 64) {
    const int64_t span = hi - lo;  // > 64, so the probes are strictly increasing
    const int64_t p = lo + span * (lane + 1) / 65;
    const int k = __popcll(__ballot(w[p] < key));  // probes 0 .. k-1 are below key
    const int64_t below = lo + span * k / 65;          // probe k-1 (k >= 1)
    const int64_t above = lo + span * (k + 1) / 65;    // probe k (k <= 63)
    if (k > 0) lo = below + 1;
    if (k < 64) hi = above;
  }
  const int64_t p = lo + lane;
  return lo + __popcll(__ballot(p < hi && w[p] < key));
}

template <bool ACC>
__global__ __launch_bounds__(TPB) void gtc_decode_tiles(const uint32_t* __restrict__ words,
                                                        const int64_t* __restrict__ count,
                                                        int64_t capacity, float tau, int64_t n,
                                                        float* __restrict__ dense) {
  __shared__ float tile[TILE];
  __shared__ int64_t range[2];
  const int64_t base = (int64_t)blockIdx.x * TILE;
  const int64_t len = n - base < TILE ? n - base : TILE;
  if (threadIdx.x < 128) {  // wave 0: the tile's first word, wave 1: the next tile's
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int64_t cnt = *count;
    cnt = cnt < 0 ? 0 : (cnt > capacity ? capacity : cnt);
    const int64_t end = base + (wv ? len : 0);
    const int64_t r = lower_bound_wave(words, cnt, (uint32_t)(end << 1), lane);
    if (lane == 0) range[wv] = r;
  }
  for (int i = threadIdx.x; i < TILE; i += TPB)
    tile[i] = (ACC && i < len) ? dense[base + i] : 0.f;
  __syncthreads();
  const int64_t lo = range[0], hi = range[1];
  for (int64_t w = lo + threadIdx.x; w < hi; w += TPB) {
    const uint32_t word = words[w];
    const int i = (int)((word >> 1) - (uint32_t)base);
    const float v = (word & 1u) ? -tau : tau;
    if ((unsigned)i >= (unsigned)len) continue;  // only for unsorted input
    if (ACC) tile[i] = tile[i] + v; else tile[i] = v;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < len; i += TPB) dense[base + i] = tile[i];
}


// Decode of one stream fused with the SGD step, for a learning rate that is
// -0.0, negative, infinite or NaN (then w - lr * 0.0 may differ from w, so
// every element is rewritten): each tile's update is built in LDS as in
// gtc_decode_tiles (accumulate = 0) and applied to every master weight of
// the tile at once, so the dense update never goes to memory; the bf16 copy
// is written for every element, as sgd_apply does.  Same results as the two
// launches, bit for bit.
template <bool ALIGNED, bool BF16>
__global__ __launch_bounds__(TPB) void gtc_decode_sgd_tiles(
    const uint32_t* __restrict__ words, const int64_t* __restrict__ count, int64_t capacity,
    float tau, int64_t n, float lr, float* __restrict__ master, bf16_t* __restrict__ wb) {
  __shared__ float tile[TILE];
  __shared__ int64_t range[2];
  const int64_t base = (int64_t)blockIdx.x * TILE;
  const int64_t len = n - base < TILE ? n - base : TILE;
  if (threadIdx.x < 128) {  // wave 0: the tile's first word, wave 1: the next tile's
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int64_t cnt = *count;
    cnt = cnt < 0 ? 0 : (cnt > capacity ? capacity : cnt);
    const int64_t end = base + (wv ? len : 0);
    const int64_t r = lower_bound_wave(words, cnt, (uint32_t)(end << 1), lane);
    if (lane == 0) range[wv] = r;
  }
  for (int i = threadIdx.x; i < TILE; i += TPB) tile[i] = 0.f;
  __syncthreads();
  const int64_t lo = range[0], hi = range[1];
  for (int64_t w = lo + threadIdx.x; w < hi; w += TPB) {
    const uint32_t word = words[w];
    const int i = (int)((word >> 1) - (uint32_t)base);
    if ((unsigned)i >= (unsigned)len) continue;  // only for unsorted input
    tile[i] = (word & 1u) ? -tau : tau;
  }
  __syncthreads();
  const double lr64 = (double)lr;
  for (int i = threadIdx.x * 4; i < len; i += TPB * 4) {
    float* mp = master + base + i;
    if (ALIGNED && i + 3 < len) {
      const float4 m = *reinterpret_cast<const float4*>(mp);
      const float4 u = *reinterpret_cast<const float4*>(tile + i);
      const float4 w = make_float4(sgd_one(m.x, u.x, lr64), sgd_one(m.y, u.y, lr64),
                                   sgd_one(m.z, u.z, lr64), sgd_one(m.w, u.w, lr64));
      *reinterpret_cast<float4*>(mp) = w;
      if (BF16) {
        uint2 b;
        b.x = (uint32_t)f32_to_bf16(w.x) | ((uint32_t)f32_to_bf16(w.y) << 16);
        b.y = (uint32_t)f32_to_bf16(w.z) | ((uint32_t)f32_to_bf16(w.w) << 16);
        *reinterpret_cast<uint2*>(wb + base + i) = b;
      }
    } else {
      for (int k = 0; k < 4 && i + k < len; ++k) {
        const float m = mp[k], u = tile[i + k];
        const float w = sgd_one(m, u, lr64);
        mp[k] = w;
        if (BF16) wb[base + i + k] = f32_to_bf16(w);
      }
    }
  }
}

// ---- aggregate of several workers' streams ----------------------------------
// Streams are the rows of words [S][capacity], each ascending in index.  A
// bounds pass finds, for every stream s and tile t, the first word of s at or
// after the tile by binary search (start[s][t], t = 0..ntiles);
// then each tile adds (1 << 16) +- 1 per word into an LDS integer per
// element (hits in the upper half, the signed sum k in the lower), and writes
// fl32(tau * k) where some word named the element.  Integer adds commute, so
// the result does not depend on the order of the streams or of the words.

__global__ __launch_bounds__(TPB) void gtc_multi_bounds(const uint32_t* __restrict__ words,
                                                        int64_t capacity,
                                                        const int64_t* __restrict__ counts,
                                                        int64_t ntiles, int64_t n,
                                                        int32_t* __restrict__ start) {
  const int s = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * TPB + threadIdx.x;
  if (t > ntiles) return;
  int64_t cnt = counts[s];
  cnt = cnt < 0 ? 0 : (cnt > capacity ? capacity : cnt);
  const int64_t first = t * TILE < n ? t * TILE : n;  // n < 2^31: the key fits
  start[(int64_t)s * (ntiles + 1) + t] =
      (int32_t)lower_bound_words(words + (int64_t)s * capacity, cnt, (uint32_t)(first << 1));
}

template <bool ACC>
__global__ __launch_bounds__(TPB) void gtc_multi_tiles(const uint32_t* __restrict__ words,
                                                       int64_t capacity,
                                                       const int64_t* __restrict__ counts,
                                                       int streams,
                                                       const int32_t* __restrict__ start,
                                                       int64_t ntiles, float tau, int64_t n,
                                                       float* __restrict__ dense) {
  __shared__ int acc[TILE];
  const int64_t t = blockIdx.x, base = t * TILE;
  const int len = (int)(n - base < TILE ? n - base : TILE);
  for (int i = threadIdx.x; i < TILE; i += TPB) acc[i] = 0;
  __syncthreads();
  for (int s = 0; s < streams; ++s) {
    int64_t cnt = counts[s];
    cnt = cnt < 0 ? 0 : (cnt > capacity ? capacity : cnt);
    const int32_t* st = start + (int64_t)s * (ntiles + 1);
    int64_t lo = st[t], hi = st[t + 1];
    lo = lo < 0 ? 0 : (lo > cnt ? cnt : lo);
    hi = hi < lo ? lo : (hi > cnt ? cnt : hi);
    const uint32_t* w = words + (int64_t)s * capacity;
    for (int64_t p = lo + threadIdx.x; p < hi; p += TPB) {
      const uint32_t word = w[p];
      const int i = (int)((word >> 1) - (uint32_t)base);
      if ((unsigned)i >= (unsigned)len) continue;  // only for malformed streams
      atomicAdd(&acc[i], (word & 1u) ? (1 << 16) - 1 : (1 << 16) + 1);
    }
  }
  __syncthreads();
  const double tau64 = (double)tau;
  for (int i = threadIdx.x; i < len; i += TPB) {
    const int v = acc[i];
    const int hits = (v + 32768) >> 16;
    const int k = v - (hits << 16);
    if (hits > 0) {
      const float q = (float)(tau64 * (double)k);
      dense[base + i] = ACC ? dense[base + i] + q : q;
    } else if (!ACC) {
      dense[base + i] = 0.f;
    }
  }
}

}  // namespace

int64_t gtc_tiles(int64_t n) { return (n + TILE - 1) / TILE; }

hipError_t gtc_encode(int64_t n, const float* g, float* r, float tau, uint32_t* words,
                      int64_t* count, uint32_t* ws_codes, int32_t* ws_tile, hipStream_t s) {
  const int64_t ntiles = gtc_tiles(n);
  if (ntiles > 0) {
    const bool aligned = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(r)) & 15) == 0;
    if (aligned)
      hipLaunchKernelGGL(gtc_update<true>, dim3((unsigned)ntiles), dim3(TPB), 0, s, n, g, r, tau,
                         ws_codes, ws_tile);
    else
      hipLaunchKernelGGL(gtc_update<false>, dim3((unsigned)ntiles), dim3(TPB), 0, s, n, g, r, tau,
                         ws_codes, ws_tile);
  }
  if (ntiles > 0 && ntiles <= OWN_PREFIX_TILES) {
    hipLaunchKernelGGL(gtc_compact_own_prefix, dim3((unsigned)ntiles), dim3(TPB), 0, s, ntiles,
                       ws_codes, ws_tile, words, count);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(gtc_scan, dim3(1), dim3(1024), 0, s, ws_tile, ntiles, count);
  if (ntiles > 0)
    hipLaunchKernelGGL(gtc_compact, dim3((unsigned)ntiles), dim3(TPB), 0, s, ws_codes, ws_tile, words);
  return hipGetLastError();
}

hipError_t gtc_decode(const uint32_t* words, const int64_t* count, int64_t capacity, float tau,
                      int64_t n, float* dense, bool accumulate, hipStream_t s) {
  const int64_t ntiles = gtc_tiles(n);
  if (ntiles == 0) return hipSuccess;
  if (accumulate)
    hipLaunchKernelGGL(gtc_decode_tiles<true>, dim3((unsigned)ntiles), dim3(TPB), 0, s, words,
                       count, capacity, tau, n, dense);
  else
    hipLaunchKernelGGL(gtc_decode_tiles<false>, dim3((unsigned)ntiles), dim3(TPB), 0, s, words,
                       count, capacity, tau, n, dense);
  return hipGetLastError();
}

}  // namespace am

namespace am {

hipError_t gtc_decode_multi(int streams, const uint32_t* words, int64_t capacity,
                            const int64_t* counts, float tau, int64_t n, float* dense,
                            bool accumulate, int32_t* ws_start, hipStream_t s) {
  const int64_t ntiles = gtc_tiles(n);
  if (ntiles == 0) return hipSuccess;
  if (streams == 0) return accumulate ? hipSuccess : fill_zero(dense, n, s);
  const unsigned bx = (unsigned)((ntiles + 1 + TPB - 1) / TPB);
  hipLaunchKernelGGL(gtc_multi_bounds, dim3(bx, (unsigned)streams), dim3(TPB), 0, s, words,
                     capacity, counts, ntiles, n, ws_start);
  if (accumulate)
    hipLaunchKernelGGL(gtc_multi_tiles<true>, dim3((unsigned)ntiles), dim3(TPB), 0, s, words,
                       capacity, counts, streams, ws_start, ntiles, tau, n, dense);
  else
    hipLaunchKernelGGL(gtc_multi_tiles<false>, dim3((unsigned)ntiles), dim3(TPB), 0, s, words,
                       capacity, counts, streams, ws_start, ntiles, tau, n, dense);
  return hipGetLastError();
}

// The same step when lr is +0.0 or positive and finite: an element no word
// names keeps its master (fl32(w - lr * 0.0) = w for non-NaN w), and its bf16
// copy already holds that master's rounding, so only the named elements are
// read and written.  Block t takes the words of tile t (found as in the
// decoder) and, for each, loads the master, applies the step and stores the
// master and its bf16 copy: about 14 bytes per sent element instead of a
// pass over all n.
template <bool BF16>
__global__ __launch_bounds__(TPB) void gtc_decode_sgd_named(
    const uint32_t* __restrict__ words, const int64_t* __restrict__ count, int64_t capacity,
    float tau, int64_t n, float lr, float* __restrict__ master, bf16_t* __restrict__ wb) {
  __shared__ int64_t range[2];
  const int64_t base = (int64_t)blockIdx.x * TILE;
  const int64_t len = n - base < TILE ? n - base : TILE;
  if (threadIdx.x < 128) {  // wave 0: the tile's first word, wave 1: the next tile's
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int64_t cnt = *count;
    cnt = cnt < 0 ? 0 : (cnt > capacity ? capacity : cnt);
    const int64_t end = base + (wv ? len : 0);
    const int64_t r = lower_bound_wave(words, cnt, (uint32_t)(end << 1), lane);
    if (lane == 0) range[wv] = r;
  }
  __syncthreads();
  const int64_t lo = range[0], hi = range[1];
  const double lr64 = (double)lr;
  for (int64_t w = lo + threadIdx.x; w < hi; w += TPB) {
    const uint32_t word = words[w];
    const int i = (int)((word >> 1) - (uint32_t)base);
    if ((unsigned)i >= (unsigned)len) continue;  // only for unsorted input
    const int64_t e = base + i;
    const float v = sgd_one(master[e], (word & 1u) ? -tau : tau, lr64);
    master[e] = v;
    if (BF16) wb[e] = f32_to_bf16(v);
  }
}

hipError_t gtc_decode_sgd(const uint32_t* words, const int64_t* count, int64_t capacity, float tau,
                          int64_t n, float lr, float* master, uint16_t* w_bf16, hipStream_t s) {
  const int64_t ntiles = gtc_tiles(n);
  if (ntiles == 0) return hipSuccess;
  const bool al = (reinterpret_cast<uintptr_t>(master) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(w_bf16) & 7) == 0;
  const uint32_t lb = __builtin_bit_cast(uint32_t, lr);
  // +0.0 or positive and finite: only the named elements change
  const bool named_only = lb == 0u || (lr > 0.f && lr <= 3.402823466e38f);
  bf16_t* wb = reinterpret_cast<bf16_t*>(w_bf16);
  const dim3 g((unsigned)ntiles), b(TPB);
  if (named_only) {
    if (wb)
      hipLaunchKernelGGL(gtc_decode_sgd_named<true>, g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
    else
      hipLaunchKernelGGL(gtc_decode_sgd_named<false>, g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
    return hipGetLastError();
  }
  if (al && wb)
    hipLaunchKernelGGL((gtc_decode_sgd_tiles<true, true>), g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
  else if (al)
    hipLaunchKernelGGL((gtc_decode_sgd_tiles<true, false>), g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
  else if (wb)
    hipLaunchKernelGGL((gtc_decode_sgd_tiles<false, true>), g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
  else
    hipLaunchKernelGGL((gtc_decode_sgd_tiles<false, false>), g, b, 0, s, words, count, capacity, tau, n, lr, master, wb);
  return hipGetLastError();
}

}  // namespace am
