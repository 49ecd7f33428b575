// libsdnn: Sparse DNN Challenge inference (Kepner et al., 2019) on MI355X (gfx950).
//
// Per layer (Sec. II batched equation, Sec. V listing):
//   z[r][j] = fma chain over the sources k of column j, ascending, of Y[r][k] * W(k, j)
//   Y'[r][j] = (z != 0) ? min(ymax, max(0, z + b[j])) : 0
// followed by dropping rows that became all zero (they stay zero) and, after the last layer, the
// categories: rows with any entry > 0 (Sec. V).
//
// Data layout in HBM
//   Activations: path 0 (widths whose tiles fit LDS, N <= 4096) keeps row-major [M][N] fp32 rows
//   and a list of live row ids; path 1 keeps feature-major tiles of 32 list positions ([N][32] fp32
//   per tile, 128 bytes per source), or after layer 0 one-byte dictionary codes in tiles of 64 or
//   128 positions, or bit tiles of 16 or 32 positions for binary inputs.
//   Weights: per layer a slot-major ELL table [K][N] of (source offset, fp32 weight), entry [s][j]
//   the s-th smallest source of output j, padded with (0, 0.0f); padding adds fma(y, 0, acc) = acc
//   exactly. Layers with 32 sources per column also get 16-bit source lists with their fp32
//   weights beside them: [32][N] u16 + [32][N] fp32 (path 1, six bytes per edge) and [4][N][8]
//   u16 + fp32 (path 0, eight per 16-byte load). With the opt-in equal-value kernels, a layer whose
//   weights and biases are all equal keeps one weight instead, and where columns share their list
//   only the representative columns' lists.
//
// Kernels (every output is the ascending-source fma chain above, so every path gives the same bits)
//   path 0: k_layer_lds (one layer; B rows staged in LDS as [k][B]), k_layers_lds (every remaining
//     layer in one launch, each workgroup's rows resident in LDS), and, opt-in, layer 0 by counts
//     of bit tiles.
//   path 1, layer 0: k_pack_bits, then k_layer_bits (or, opt-in for one-weight layers,
//     k_count_dict + k_layer_count: adder-tree counts of set source bits, decoded by a
//     dictionary); non-binary inputs take k_to_fm + k_layer_gfm.
//   path 1, later layers: k_layer_gfm_u8 (code tiles in), k_layer_gfm (fp32 tiles in),
//     k_layer_gfm_small (at most 8 tiles, whole chains in flight). Workgroups are mapped so that
//     each XCD gathers from its own tile, resident in its L2.
//   Between layers: liveness words per tile (spread over cache lines, or per-workgroup partial
//   words), k_compact (stable compaction of the live list), k_repack / k_repack_u8 (regroup live
//   positions into fewer tiles), k_final_ids.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <type_traits>
#include <thread>
#include <unordered_map>
#include <vector>

#include "sdnn.h"

namespace {

thread_local std::string g_err;

sdnn_status fail(sdnn_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

constexpr int kMaxNeurons = 65536;
constexpr int kMaxLayers = 1000000;
constexpr int kMaxDegree = 4096;
constexpr int kLdsTileBytes = 128 * 1024;  // activation tile budget per workgroup
constexpr int kGfmOutputs = 64;            // outputs per work item of k_layer_gfm
constexpr int kPollEvery = 16;             // layers between live-count read-backs
constexpr int64_t kEncodeMinRows = 2048;   // live rows from which a fp32-input layer tries codes

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Run f(i) for i in [0, n) on up to 16 host threads (used for host-side validation and packing).
template <class F>
void parallel_for(int32_t n, F f) {
  const int32_t nt = std::max<int32_t>(1, std::min<int32_t>({n, 16, (int32_t)std::max(1u, std::thread::hardware_concurrency())}));
  if (nt == 1) {
    for (int32_t i = 0; i < n; ++i) f(i);
    return;
  }
  std::atomic<int32_t> next{0};
  std::vector<std::thread> th;
  for (int32_t t = 0; t < nt; ++t)
    th.emplace_back([&]() {
      for (int32_t i = next++; i < n; i = next++) f(i);
    });
  for (auto &x : th) x.join();
}

// ------------------------------------------------------------------------------------------------
// Device code

__device__ __forceinline__ float activate(float z, float b, float ymax) {
  // Sec. V loop: the bias goes only to nonzero products, then the result is clamped to [0, ymax].
  // Zeros come out as +0: for z != 0 the sum t is never -0 (x + y = -0 needs x = y = -0, and a sum
  // of nonzero values that is zero is +0), so the median of (t, +0, ymax), ymax > 0, is +0 for t <= 0.
  const float t = __builtin_amdgcn_fmed3f(z + b, 0.0f, ymax);
  return z == 0.0f ? 0.0f : t;
}

// Keeps the compiler from moving memory accesses across this point (no instruction is emitted):
// pins the issue order of software-pipelined loads.
__device__ __forceinline__ void mem_fence_compiler() { asm volatile("" ::: "memory"); }

// Sets bits m in a liveness mask word that many workgroups report to. They report mostly the same
// rows, and hundreds of atomics on one word from workgroups that finish together serialize (several
// us per launch), so only bits not yet set go through an atomic. Within a layer bits are only ever
// set, so a set bit read here is final; a stale read only costs an atomic.
// Liveness words of large layers. Device-scope atomics on one 128-byte line serialize across
// workgroups (2048 workgroups of a launch ORing into one line: tens of us), while atomics on
// different lines proceed in parallel. So mask word t of such a layer is spread over kSpread words
// in lines of their own, spread[(t * kSpread + g) * kLineWords] with g taken from the workgroup
// index, and k_spread_to_masks ORs them into masks[t] before a compaction reads it.
constexpr int kSpread = 8, kLineWords = 32;
__device__ __forceinline__ void or_mask(unsigned *masks, unsigned *spread, int t, unsigned m) {
  if (spread)
    atomicOr(&spread[((size_t)t * kSpread + ((blockIdx.x >> 3) & (kSpread - 1))) * kLineWords], m);
  else
    atomicOr(&masks[t], m);
}

// Ties four values to this point of the instruction stream (no instruction is emitted): the
// computations producing them are scheduled before it.
__device__ __forceinline__ void pin4(float &a, float &b, float &c, float &d) {
  asm volatile("" : "+v"(a), "+v"(b), "+v"(c), "+v"(d));
}

// 16-byte store that streams past the L2 (the data is read by the next kernel, not this one).
__device__ __forceinline__ void store_stream(float4 *p, float4 v) {
  typedef float v4f __attribute__((ext_vector_type(4)));
  const v4f x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<v4f *>(p));
}

__device__ __forceinline__ void store_stream(uint4 *p, uint4 v) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  const v4u x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<v4u *>(p));
}

// 16-byte nontemporal load, for data that is read exactly once (the input rows). Data that other
// workgroups read again (weights, activation tiles) takes plain loads, which measure faster.
__device__ __forceinline__ float4 load_stream_f4(const float4 *p) {
  typedef float v4f __attribute__((ext_vector_type(4)));
  const v4f x = __builtin_nontemporal_load(reinterpret_cast<const v4f *>(p));
  return make_float4(x[0], x[1], x[2], x[3]);
}


// Raw buffer resource over `bytes` bytes at p (stride 0, offsets in bytes): an access past the end
// reads zeros. The third dword is the gfx9 default format word.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *p, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ bool any_nonzero(float4 v) {
  return v.x != 0.0f || v.y != 0.0f || v.z != 0.0f || v.w != 0.0f;
}

// misc[0]: a layer-0 input is not 0 or 1; misc[kOverflowSlot]: the value dictionary is full;
// misc[3]: first live count of a uniform layer 0; misc[kNposSlot + i]: positions in live list i.
// The value dictionary's initial state (its layout is described with dict_code below): code 0 is
// +0.0, whose key 0 sits in its hash slot 0; every other slot is free and the next code is 1.
constexpr unsigned kDictEmpty = 0x7fc00000u;
constexpr unsigned kNoCode = 0xffffffffu;
constexpr int kDictSlots = 256;       // codes
constexpr int kDictHashSlots = 1024;  // hash table slots
constexpr int kDictKey = kDictSlots, kDictCode = kDictKey + kDictHashSlots, kDictNext = kDictCode + kDictHashSlots,
              kDictWords = kDictNext + 256;
// The two dictionaries: one-byte codes (above) and two-byte codes (4096 values, for layer inputs
// that take more than 256). Words: val[kSlots] | key[kHash] | code[kHash] | next; the hash slot of
// a key is bits kHashShift.. of its 24-bit multiplicative hash, the LDS cache set bits kCacheShift..
template <int CB> struct DictShape;
template <> struct DictShape<1> {
  static constexpr int kSlots = kDictSlots, kHash = kDictHashSlots, kHashShift = 14, kCache = 1024, kCacheShift = 12;
};
template <> struct DictShape<2> {
  static constexpr int kSlots = 4096, kHash = 16384, kHashShift = 10, kCache = 4096, kCacheShift = 10;
};
template <int CB> __host__ __device__ constexpr int dict_key_off() { return DictShape<CB>::kSlots; }
template <int CB> __host__ __device__ constexpr int dict_code_off() { return dict_key_off<CB>() + DictShape<CB>::kHash; }
template <int CB> __host__ __device__ constexpr int dict_next_off() { return dict_code_off<CB>() + DictShape<CB>::kHash; }
template <int CB> __host__ __device__ constexpr int dict_words() { return dict_next_off<CB>() + 256; }
static_assert(dict_words<1>() == kDictWords, "one-byte dictionary layout");
template <int CB = 1>
__device__ __forceinline__ void dict_init(unsigned *dict, int t, int nt) {
  constexpr int KEY = dict_key_off<CB>(), CODE = dict_code_off<CB>(), NEXT = dict_next_off<CB>();
  for (int i = t; i <= NEXT; i += nt)
    dict[i] = i < KEY ? 0u : i < CODE ? (i == KEY ? 0u : kDictEmpty) : i < NEXT ? (i == CODE ? 0u : kNoCode) : 1u;
}

constexpr int kOverflowSlot = 2;
constexpr int kNposSlot = 4;
__global__ void k_init(int *__restrict__ ids, unsigned *__restrict__ masks, unsigned *__restrict__ masks2,
                       unsigned *__restrict__ masks3, int *__restrict__ rownz, int *__restrict__ counts,
                       int *__restrict__ misc, unsigned *__restrict__ dict, int M, int L,
                       unsigned *__restrict__ spread, size_t spread_words) {
  const int st = gridDim.x * blockDim.x;
  // value dictionary (see dict_code): code 0 is +0.0, whose key 0 sits in its hash slot 0; every
  // other slot is free and the next code is 1
  if (blockIdx.x == 0) dict_init(dict, threadIdx.x, blockDim.x);
  if (blockIdx.x == 0 && threadIdx.x < 8) misc[threadIdx.x] = (threadIdx.x == kNposSlot) ? M : 0;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < M; i += st) {
    ids[i] = i;
    masks[i] = 0u;
    masks2[i] = 0u;
    masks3[i] = 0u;
    rownz[i] = 0;
  }
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i <= L; i += st) counts[i] = (i == 0) ? M : 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < spread_words; i += st) spread[i] = 0u;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_sum(int v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  return v;
}

// Stable compaction over per-tile liveness masks: bit b of masks[t] says that list position
// t*B + b is live. ids_out = the live ids in list order, src_out (unless null) = their positions in
// the input list, *count_out (and *count_out2 unless null) = their number. The masks are cleared for
// the next layer. One workgroup of 1024 threads; tiles are taken 4096 at a time: an exclusive scan
// of their popcounts gives each tile's output offset, then every position is placed.
constexpr int kCompactTiles = 4096;
// masks[t] = OR of the spread words of tile t (see or_mask) for the tiles of the first *npos list
// positions; the spread words are zeroed for the next large layer.
__global__ __launch_bounds__(256) void k_spread_to_masks(unsigned *__restrict__ spread, const int *__restrict__ npos,
                                                         unsigned *__restrict__ masks) {
  const int nt = (*npos + 31) / 32;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < nt; t += gridDim.x * blockDim.x) {
    unsigned m = 0u;
#pragma unroll
    for (int g = 0; g < kSpread; ++g) {
      unsigned *w = &spread[((size_t)t * kSpread + g) * kLineWords];
      m |= *w;
      *w = 0u;
    }
    masks[t] = m;
  }
}

// With notify set, thread 0 finally stores (tag << 40) | (flags << 32) | count into that word of
// coherent host memory, flags = bit 0: misc[0] (a layer-0 input is not 0 or 1), bit 1:
// misc[kOverflowSlot] (the value dictionary is full); the host waits on it instead of a copy and a
// stream synchronization.
__global__ __launch_bounds__(1024) void k_compact(unsigned *__restrict__ masks, int B, const int *__restrict__ ids_in,
                                                  int *__restrict__ ids_out, int *__restrict__ src_out,
                                                  const int *__restrict__ count_in, int *__restrict__ count_out,
                                                  int *__restrict__ count_out2, const int *__restrict__ misc,
                                                  unsigned long long *__restrict__ notify, unsigned long long tag) {
  __shared__ int toff[kCompactTiles];
  __shared__ unsigned tmask[kCompactTiles];
  __shared__ int wsum[16];
  const int R = *count_in;
  const int ntiles = (R + B - 1) / B;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int base = 0;
  for (int c0 = 0; c0 < ntiles; c0 += kCompactTiles) {
    unsigned m[4];
    int local = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = c0 + tid * 4 + q;
      m[q] = 0u;
      if (t < ntiles) {
        m[q] = masks[t];
        masks[t] = 0u;
      }
      local += __popc(m[q]);
    }
    const int incl = wave_inclusive_sum(local, lane);
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int off = 0, total = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const int x = wsum[w];
      off += (w < wave) ? x : 0;
      total += x;
    }
    int excl = base + off + incl - local;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      toff[tid * 4 + q] = excl;
      tmask[tid * 4 + q] = m[q];
      excl += __popc(m[q]);
    }
    __syncthreads();
    const int p_end = min(R, (c0 + kCompactTiles) * B);
    for (int p = c0 * B + tid; p < p_end; p += 1024) {
      const int tl = p / B - c0, b = p % B;
      const unsigned mk = tmask[tl];
      if ((mk >> b) & 1u) {
        const unsigned below = b == 0 ? 0u : (mk & (0xffffffffu >> (32 - b)));
        const int o = toff[tl] + __popc(below);
        ids_out[o] = ids_in[p];
        if (src_out) src_out[o] = p;
      }
    }
    base += total;
    __syncthreads();
  }
  if (tid == 0) {
    *count_out = base;
    if (count_out2) *count_out2 = base;
    if (notify) {
      const unsigned long long flags = (misc[0] != 0 ? 1ull : 0ull) | (misc[kOverflowSlot] != 0 ? 2ull : 0ull);
      __hip_atomic_store(notify, (tag << 40) | (flags << 32) | (unsigned long long)(unsigned)base, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

// Zeros into the 128-byte segments of fp32 tiles [0, (*npos + 31) / 32) whose seglive bit is clear
// (segments that a producer skipped because all their rows are zero), for readers that take the
// tiles as they are. 8 lanes write one segment.
__global__ __launch_bounds__(256) void k_fill_dead(float *__restrict__ fm, int N, const unsigned *__restrict__ seglive,
                                                   const int *__restrict__ npos) {
  const int ntiles = (*npos + 31) / 32;
  const int NW = (N + 31) / 32;
  const size_t items = (size_t)ntiles * N * 8;
  for (size_t it = blockIdx.x * (size_t)blockDim.x + threadIdx.x; it < items; it += (size_t)gridDim.x * blockDim.x) {
    const int q = (int)(it & 7);
    const size_t seg = it >> 3;
    const int k = (int)(seg % N);
    const size_t t = seg / N;
    if (!((seglive[t * NW + (k >> 5)] >> (k & 31)) & 1u))
      reinterpret_cast<float4 *>(fm + seg * 32)[q] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
}

// Copy list positions pos[0..n) of feature-major tiles out as rows: out[i][k] = fm at position
// pos[i], source k.
__global__ __launch_bounds__(256) void k_gather_rows(const float *__restrict__ fm, int N, const int *__restrict__ pos,
                                                     int n, float *__restrict__ out) {
  const size_t items = (size_t)n * N;
  for (size_t it = blockIdx.x * (size_t)blockDim.x + threadIdx.x; it < items; it += (size_t)gridDim.x * blockDim.x) {
    const int i = (int)(it / N), k = (int)(it % N);
    const int p = pos[i];
    out[it] = fm[((size_t)(p >> 5) * N + k) * 32 + (p & 31)];
  }
}

__global__ void k_final_ids(const int *__restrict__ ids, const int *__restrict__ count, long long *__restrict__ out) {
  const int R = *count;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < R; i += gridDim.x * blockDim.x) out[i] = ids[i];
}

// Split a tile's outputs into chunks so that small live counts still spread over the whole grid:
// with many tiles every work item is a whole tile; with few, each tile's outputs are divided.
struct Chunking {
  int nchunks, rounds_per_chunk;
};

// Tile of item w when whole tiles are the items and tpg consecutive tiles share one code group:
// the tpg tiles of a group go to workgroups of the same XCD (workgroup x runs on XCD x % 8), so the
// parts that they write of each code segment meet in that XCD's L2. A bijection of
// [0, gridDim * ceil(n / gridDim)) onto itself; needs gridDim % (8 * tpg) == 0.
__device__ __forceinline__ int code_group_tile(int w, int tpg) {
  const int per_iter = gridDim.x;
  const int k = w / per_iter, x = w % per_iter;
  const int xcd = x & 7, sl = x >> 3;
  const int g = k * (per_iter / tpg) + xcd + 8 * (sl / tpg);
  return tpg * g + sl % tpg;
}
__device__ __forceinline__ Chunking chunking(int ntiles, int rounds, int min_chunks = 1) {
  int nchunks = ntiles > 0 ? (int)gridDim.x / ntiles : 1;
  nchunks = max(min_chunks, min(nchunks, rounds));
  nchunks = min(nchunks, rounds);
  const int rpc = (rounds + nchunks - 1) / nchunks;
  return {(rounds + rpc - 1) / rpc, rpc};
}

// LDS reads in flight ahead of the fmas in the LDS-tile kernels' 32-term chains
#ifndef SDNN_LDS_AHEAD
#define SDNN_LDS_AHEAD 6
#endif
constexpr int kLdsAhead = SDNN_LDS_AHEAD;

// One layer with the activation tile staged in LDS. B rows per tile (4 <= B <= 32, a multiple of 4);
// blockDim 1024. KC is the compile-time ELL width (0: use the runtime K). With cols set (one-weight
// layers through ell16 only), the ncols columns cols[p] alone are computed and written, their
// source lists in ell16 as [4][ncols][8]; the other columns equal one of them (see k_layer_gfm).
// With place set, neuron k is staged at tile row place[k] and ell16 holds tile rows (placed
// sources; see bank_placement), which only changes which LDS banks the reads fall in.
template <int B, int KC>
__global__ __launch_bounds__(1024) void k_layer_lds(const float *__restrict__ yin, float *__restrict__ yout, int N,
                                                    const int2 *__restrict__ ell, int K,
                                                    const uint4 *__restrict__ ell16, const float *__restrict__ w8,
                                                    float wc,
                                                    const float *__restrict__ bias, float ymax,
                                                    const int *__restrict__ ids, const int *__restrict__ count,
                                                    unsigned *__restrict__ masks, int *__restrict__ rownz,
                                                    const int *__restrict__ cols, int ncols,
                                                    const unsigned short *__restrict__ place) {
  extern __shared__ float4 smem[];
  const char *tile = reinterpret_cast<const char *>(smem);
  float *tilef = reinterpret_cast<float *>(smem);
  __shared__ int rowlive[B];
  __shared__ int rowany[B];
  constexpr int LPO = B / 4;    // lanes per output, 4 rows each
  constexpr int OPW = 64 / LPO; // outputs per wave instruction
  const int R = *count;
  const int ntiles = (R + B - 1) / B;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int quad = lane % LPO, jl = lane / LPO;
  const int per_round = nw * OPW;
  const int rounds = (ncols + per_round - 1) / per_round;
  const Chunking ch = chunking(ntiles, rounds);
  const int items = ntiles * ch.nchunks;
  if (tid < B) {
    rowlive[tid] = 0;
    rowany[tid] = 0;
  }
  for (int w = blockIdx.x; w < items; w += gridDim.x) {
    const int t = w / ch.nchunks, c = w % ch.nchunks;
    const int p0 = t * B;
    const int nvalid = min(B, R - p0);
    const bool count_nz = rownz != nullptr && c == 0;
    // ---- stage rows ids[p0 .. p0+nvalid) as tile[k][b]; missing rows are zero
    if ((N & 3) == 0) {
      const int NQ = N >> 2;
      const int nitems = NQ * (B / 4);
      for (int it = tid; it < nitems; it += blockDim.x) {
        const int bq = it % (B / 4), q = it / (B / 4);
        float4 v[4];
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const int b = bq * 4 + c4;
          v[c4] = (b < nvalid) ? reinterpret_cast<const float4 *>(yin + (size_t)ids[p0 + b] * N)[q]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        // neuron k goes to tile row place[k] (k itself without a placement)
        int rk[4];
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) rk[c4] = place ? (int)place[4 * q + c4] : 4 * q + c4;
        float *dst = tilef + bq * 4;
        *reinterpret_cast<float4 *>(dst + (size_t)rk[0] * B) = make_float4(v[0].x, v[1].x, v[2].x, v[3].x);
        *reinterpret_cast<float4 *>(dst + (size_t)rk[1] * B) = make_float4(v[0].y, v[1].y, v[2].y, v[3].y);
        *reinterpret_cast<float4 *>(dst + (size_t)rk[2] * B) = make_float4(v[0].z, v[1].z, v[2].z, v[3].z);
        *reinterpret_cast<float4 *>(dst + (size_t)rk[3] * B) = make_float4(v[0].w, v[1].w, v[2].w, v[3].w);
        if (count_nz) {
#pragma unroll
          for (int c4 = 0; c4 < 4; ++c4)
            if (any_nonzero(v[c4])) rowany[bq * 4 + c4] = 1;
        }
      }
    } else {
      for (int it = tid; it < N * B; it += blockDim.x) {
        const int b = it % B, k = it / B;
        const float v = (b < nvalid) ? yin[(size_t)ids[p0 + b] * N + k] : 0.0f;
        tilef[(size_t)(place ? (int)place[k] : k) * B + b] = v;
        if (count_nz && v != 0.0f) rowany[b] = 1;
      }
    }
    __syncthreads();
    // ---- compute: lane (quad, jl) owns rows 4*quad..4*quad+3 of output j
    int row[4];
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      const int b = quad * 4 + c4;
      row[c4] = (b < nvalid) ? ids[p0 + b] : -1;
    }
    const int qoff = quad * 16;
    int live_mask = 0;
    const int r_end = min(rounds, (c + 1) * ch.rounds_per_chunk);
    for (int r = c * ch.rounds_per_chunk; r < r_end; ++r) {
      const int j = r * per_round + wave * OPW + jl;  // output position (the column without cols)
      if (j >= ncols) continue;
      const int col = cols ? cols[j] : j;
      float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, a3 = 0.0f;
      // ELL is slot-major ([s][j]): for a given slot the lanes of a wave read consecutive entries.
      // Terms go in groups of 8 in ascending source order; with KC known, the next group's
      // entries are loaded (unconditionally, so no branch delays the wait counts) while the
      // current group's LDS reads and fma chain run.
      const int2 *ej = ell + j;
      if (ell16) {
        // 32 sources per column, eight per 16-byte load ([4][N][8] u16), with their weights in the
        // same grouping (w8, two 16-byte loads per eight) or the layer's one weight wc; all loads
        // are in flight before the first group's LDS reads
        uint4 ix[4];
        float4 wq[8];
#pragma unroll
        for (int g = 0; g < 4; ++g) ix[g] = ell16[(size_t)g * ncols + j];
        if (w8) {
          const float4 *w4 = reinterpret_cast<const float4 *>(w8);
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            wq[2 * g] = w4[((size_t)g * ncols + j) * 2];
            wq[2 * g + 1] = w4[((size_t)g * ncols + j) * 2 + 1];
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) wq[i] = make_float4(wc, wc, wc, wc);
        }
        // the 32 terms in order, each slot's LDS read issued kLdsAhead slots before its fmas (a
        // rotating buffer, so reads stay in flight across the groups of eight)
        auto src_of = [&](int sl) {
          const uint4 &g = ix[sl / 8];
          const unsigned pr = (sl % 8) < 2 ? g.x : (sl % 8) < 4 ? g.y : (sl % 8) < 6 ? g.z : g.w;
          return (sl & 1) ? (pr >> 16) : (pr & 0xffffu);
        };
        auto w_of = [&](int sl) {
          const float4 &q = wq[sl / 4];
          return (sl % 4) == 0 ? q.x : (sl % 4) == 1 ? q.y : (sl % 4) == 2 ? q.z : q.w;
        };
        auto rd = [&](int sl) { return *reinterpret_cast<const float4 *>(tile + src_of(sl) * (unsigned)(B * 4) + qoff); };
        float4 buf[kLdsAhead];
#pragma unroll
        for (int q = 0; q < kLdsAhead; ++q) buf[q] = rd(q);
#pragma unroll
        for (int sl = 0; sl < 32; ++sl) {
          const float4 v = buf[sl % kLdsAhead];
          if (sl + kLdsAhead < 32) buf[sl % kLdsAhead] = rd(sl + kLdsAhead);
          const float w = w_of(sl);
          a0 = fmaf(v.x, w, a0);
          a1 = fmaf(v.y, w, a1);
          a2 = fmaf(v.z, w, a2);
          a3 = fmaf(v.w, w, a3);
        }
      } else if constexpr (KC > 0) {
        static_assert(KC % 8 == 0, "KC must be a multiple of 8");
        int2 cur[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) cur[q] = ej[(size_t)q * N];
#pragma unroll 1
        for (int g = 0; g < KC - 8; g += 8) {
          int2 nxt[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) nxt[q] = ej[(size_t)(g + 8 + q) * N];
          float4 v[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] = *reinterpret_cast<const float4 *>(tile + cur[q].x + qoff);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float wv = __int_as_float(cur[q].y);
            a0 = fmaf(v[q].x, wv, a0);
            a1 = fmaf(v[q].y, wv, a1);
            a2 = fmaf(v[q].z, wv, a2);
            a3 = fmaf(v[q].w, wv, a3);
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) cur[q] = nxt[q];
        }
        float4 v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = *reinterpret_cast<const float4 *>(tile + cur[q].x + qoff);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float wv = __int_as_float(cur[q].y);
          a0 = fmaf(v[q].x, wv, a0);
          a1 = fmaf(v[q].y, wv, a1);
          a2 = fmaf(v[q].z, wv, a2);
          a3 = fmaf(v[q].w, wv, a3);
        }
      } else {
        for (int s2 = 0; s2 < K; ++s2) {
          const int2 p = ej[(size_t)s2 * N];
          const float4 v = *reinterpret_cast<const float4 *>(tile + p.x + qoff);
          const float wv = __int_as_float(p.y);
          a0 = fmaf(v.x, wv, a0);
          a1 = fmaf(v.y, wv, a1);
          a2 = fmaf(v.z, wv, a2);
          a3 = fmaf(v.w, wv, a3);
        }
      }
      const float bj = bias[col];
      const float y[4] = {activate(a0, bj, ymax), activate(a1, bj, ymax), activate(a2, bj, ymax),
                          activate(a3, bj, ymax)};
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        if (row[c4] >= 0) {
          yout[(size_t)row[c4] * N + col] = y[c4];
          if (y[c4] > 0.0f) live_mask |= 1 << c4;
        }
      }
    }
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4)
      if (live_mask & (1 << c4)) rowlive[quad * 4 + c4] = 1;
    __syncthreads();
    if (tid < 64) {
      const unsigned long long m = __ballot(tid < nvalid && rowlive[tid] != 0);
      if (tid == 0 && m) atomicOr(&masks[t], (unsigned)m);
      if (count_nz && tid < nvalid && rowany[tid]) rownz[ids[p0 + tid]] = 1;
    }
    if (tid < B) {
      rowlive[tid] = 0;
      rowany[tid] = 0;
    }
    __syncthreads();
  }
}

// Device view of one layer for kernels that run several layers in one launch.
struct LayerPtr {
  const int2 *ell;     // slot-major ELL, offsets in units of 1 << ell_shift bytes per source
  const uint4 *ell16;  // layer with 32 sources per column: [4][D][8] u16 sources, else null
  const float *w8;     // with ell16: the weights in the same grouping, [4][D][8] fp32; null for a
                       // uniform layer (weight w)
  const float *bias;
  const int *cols;     // with ell16: the D columns computed (null: all N, D = N)
  float w;             // the weight of a one-weight layer
  int K;
  int D;
};

// RPL consecutive fp32 rows of one source, read or written as one LDS access
template <int RPL>
__device__ __forceinline__ void lds_rows_load(const char *p, float (&v)[RPL]) {
  if constexpr (RPL == 4) {
    const float4 t = *reinterpret_cast<const float4 *>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (RPL == 2) {
    const float2 t = *reinterpret_cast<const float2 *>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = *reinterpret_cast<const float *>(p);
  }
}
template <int RPL>
__device__ __forceinline__ void lds_rows_store(float *p, const float (&v)[RPL]) {
  if constexpr (RPL == 4) *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  else if constexpr (RPL == 2) *reinterpret_cast<float2 *>(p) = make_float2(v[0], v[1]);
  else *p = v[0];
}

// Layers [l0, L) of the live rows listed in ids (count *count), in one launch: workgroup g keeps
// list positions [gB, gB + B) in LDS across all the layers, as two tiles [k][B] (the layer's input
// and its output), so between layers nothing goes through global memory and nothing waits for other
// workgroups (rows are independent, Sec. V). A lane holds RPL = min(B, 4) rows: lane = (quad = lane
// % (B/RPL): rows RPL quad .. RPL quad + RPL - 1, output slot lane / (B/RPL)); each term is one LDS
// read of RPL rows (16, 8 or 4 bytes) and RPL fmas, in ascending source order as everywhere. Small
// B spreads a short list over more CUs. After every layer the workgroup adds its live rows to
// counts[l + 1] and stops once none is left (rows that die stay dead). Rows still live after layer
// L - 1 are written to yout (row-major, by row id) and marked in masks (one bit per list position)
// for the final compaction. A layer with cols computes only those columns (the others are never
// read: the next layer's sources are representatives, and final rows are expanded on the host).
// Dynamic LDS: 2 * N * B floats.
template <int B>
__global__ __launch_bounds__(1024) void k_layers_lds(const float *__restrict__ yin, float *__restrict__ yout, int N,
                                                     const LayerPtr *__restrict__ lp, int l0, int L, float ymax,
                                                     const int *__restrict__ ids, const int *__restrict__ count,
                                                     int *__restrict__ counts, unsigned *__restrict__ masks,
                                                     int ell_shift) {
  static_assert(B == 1 || B == 2 || B == 4 || B == 8 || B == 16, "lanes hold up to 4 rows, at most 4 lanes per output");
  constexpr int RPL = B < 4 ? B : 4;
  extern __shared__ float4 smem[];
  __shared__ unsigned livebits[2];
  float *ta = reinterpret_cast<float *>(smem);
  float *tc = ta + (size_t)N * B;
  const int R = *count;
  const int p0 = blockIdx.x * B;
  if (p0 >= R) return;  // uniform over the workgroup
  const int nvalid = min(B, R - p0);
  const unsigned valid = (1u << nvalid) - 1u;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  constexpr int LPO = B / RPL, OPW = 64 / LPO;
  const int quad = lane % LPO, jl = lane / LPO;
  const int per_round = nw * OPW;
  // stage the rows as ta[k][b] (reads run along k); positions past the list are zero
  for (int it = tid; it < N * B; it += blockDim.x) {
    const int b = it / N, k = it % N;
    ta[(size_t)k * B + b] = b < nvalid ? yin[(size_t)ids[p0 + b] * N + k] : 0.0f;
  }
  unsigned lb = valid;
  int l = l0;
  for (; l < L; ++l) {
    const LayerPtr P = lp[l];
    // livebits[l & 1] was last read before the barrier at the top of layer l - 1
    if (tid == 0) livebits[l & 1] = 0u;
    __syncthreads();  // ta is complete, and every read of tc (the layer before's input) is done
    unsigned lm = 0u;
    const char *tq = reinterpret_cast<const char *>(ta) + quad * (RPL * 4);
    const int ncols = P.ell16 ? P.D : N;
    const int rounds = (ncols + per_round - 1) / per_round;
    for (int r = 0; r < rounds; ++r) {
      const int jp = r * per_round + wave * OPW + jl;
      if (jp >= ncols) break;
      const int j = P.cols ? P.cols[jp] : jp;
      float a[RPL];
#pragma unroll
      for (int c = 0; c < RPL; ++c) a[c] = 0.0f;
      if (P.ell16) {
        // 32 sources, eight per 16-byte load ([4][D][8] u16), and their weights (eight per two
        // 16-byte loads from w8, or the layer's one weight); every load in flight first
        uint4 ix[4];
        float4 wq[8];
#pragma unroll
        for (int g = 0; g < 4; ++g) ix[g] = P.ell16[(size_t)g * ncols + jp];
        if (P.w8) {
          const float4 *w4 = reinterpret_cast<const float4 *>(P.w8);
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            wq[2 * g] = w4[((size_t)g * ncols + jp) * 2];
            wq[2 * g + 1] = w4[((size_t)g * ncols + jp) * 2 + 1];
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) wq[i] = make_float4(P.w, P.w, P.w, P.w);
        }
        // the 32 terms in order, each slot's LDS read issued kLdsAhead slots before its fmas
        auto src_of = [&](int sl) {
          const uint4 &g = ix[sl / 8];
          const unsigned pr = (sl % 8) < 2 ? g.x : (sl % 8) < 4 ? g.y : (sl % 8) < 6 ? g.z : g.w;
          return (sl & 1) ? (pr >> 16) : (pr & 0xffffu);
        };
        auto w_of = [&](int sl) {
          const float4 &q = wq[sl / 4];
          return (sl % 4) == 0 ? q.x : (sl % 4) == 1 ? q.y : (sl % 4) == 2 ? q.z : q.w;
        };
        float buf[kLdsAhead][RPL];
#pragma unroll
        for (int q = 0; q < kLdsAhead; ++q) lds_rows_load<RPL>(tq + src_of(q) * (unsigned)(B * 4), buf[q]);
#pragma unroll
        for (int sl = 0; sl < 32; ++sl) {
          float v[RPL];
#pragma unroll
          for (int c = 0; c < RPL; ++c) v[c] = buf[sl % kLdsAhead][c];
          if (sl + kLdsAhead < 32) lds_rows_load<RPL>(tq + src_of(sl + kLdsAhead) * (unsigned)(B * 4), buf[sl % kLdsAhead]);
          const float w = w_of(sl);
#pragma unroll
          for (int c = 0; c < RPL; ++c) a[c] = fmaf(v[c], w, a[c]);
        }
      } else {
        for (int sl = 0; sl < P.K; ++sl) {
          const int2 e = P.ell[(size_t)sl * N + j];
          float v[RPL];
          lds_rows_load<RPL>(tq + ((unsigned)e.x >> ell_shift) * (unsigned)(B * 4), v);
          const float wv = __int_as_float(e.y);
#pragma unroll
          for (int c = 0; c < RPL; ++c) a[c] = fmaf(v[c], wv, a[c]);
        }
      }
      const float bj = P.bias[j];
      float y[RPL];
      unsigned bits = 0u;
#pragma unroll
      for (int c = 0; c < RPL; ++c) {
        y[c] = activate(a[c], bj, ymax);
        bits |= (y[c] > 0.0f ? 1u : 0u) << c;
      }
      lds_rows_store<RPL>(tc + (size_t)j * B + quad * RPL, y);
      lm |= bits << (RPL * quad);
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) lm |= __shfl_xor(lm, d, 64);
    if (lane == 0 && lm) atomicOr(&livebits[l & 1], lm);
    __syncthreads();
    lb = livebits[l & 1] & valid;
    if (tid == 0 && lb) atomicAdd(&counts[l + 1], __popc(lb));
    float *t = ta;
    ta = tc;
    tc = t;
    if (!lb) break;
  }
  if (l == L && lb) {
    // ta holds the output of layer L - 1
    for (int it = tid; it < N * B; it += blockDim.x) {
      const int b = it / N, k = it % N;
      if ((lb >> b) & 1u) yout[(size_t)ids[p0 + b] * N + k] = ta[(size_t)k * B + b];
    }
    if (tid < B && ((lb >> tid) & 1u)) atomicOr(&masks[(p0 + tid) >> 5], 1u << ((p0 + tid) & 31));
  }
}

// Copy live rows into feature-major tiles of FMR rows: fm[t][k][b] = Y[ids[t*FMR + b]][k], zero
// for positions past the live count.
template <int FMR>
__global__ __launch_bounds__(256) void k_to_fm(const float *__restrict__ yin, float *__restrict__ fm, int N,
                                               const int *__restrict__ ids, const int *__restrict__ count,
                                               int *__restrict__ rownz) {
  const int R = *count;
  const int ntiles = (R + FMR - 1) / FMR;
  const size_t st = (size_t)gridDim.x * blockDim.x;
  if ((N & 3) == 0) {
    const int NQ = N >> 2;
    const size_t items = (size_t)ntiles * NQ * (FMR / 4);
    for (size_t it = blockIdx.x * (size_t)blockDim.x + threadIdx.x; it < items; it += st) {
      const int bq = (int)(it % (FMR / 4));
      const size_t rest = it / (FMR / 4);
      const int q = (int)(rest % NQ);
      const int t = (int)(rest / NQ);
      float4 v[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int p = t * FMR + bq * 4 + c;
        v[c] = (p < R) ? reinterpret_cast<const float4 *>(yin + (size_t)ids[p] * N)[q] : make_float4(0.f, 0.f, 0.f, 0.f);
        if (rownz && p < R && any_nonzero(v[c]) && !rownz[ids[p]]) rownz[ids[p]] = 1;
      }
      float4 *dst = reinterpret_cast<float4 *>(fm + ((size_t)t * N + 4 * q) * FMR + bq * 4);
      dst[0] = make_float4(v[0].x, v[1].x, v[2].x, v[3].x);
      dst[FMR / 4] = make_float4(v[0].y, v[1].y, v[2].y, v[3].y);
      dst[2 * (FMR / 4)] = make_float4(v[0].z, v[1].z, v[2].z, v[3].z);
      dst[3 * (FMR / 4)] = make_float4(v[0].w, v[1].w, v[2].w, v[3].w);
    }
  } else {
    const size_t items = (size_t)ntiles * N * FMR;
    for (size_t it = blockIdx.x * (size_t)blockDim.x + threadIdx.x; it < items; it += st) {
      const int b = (int)(it % FMR);
      const size_t rest = it / FMR;
      const int k = (int)(rest % N);
      const int t = (int)(rest / N);
      const int p = t * FMR + b;
      const float v = (p < R) ? yin[(size_t)ids[p] * N + k] : 0.0f;
      fm[((size_t)t * N + k) * FMR + b] = v;
      if (rownz && v != 0.0f && !rownz[ids[p]]) rownz[ids[p]] = 1;
    }
  }
}

// Weight layouts read by the global-tile kernels:
//   kWEll:  a layer of any width K: the slot-major ELL of (source offset, weight bits), K from the
//           launch (the general fallback);
//   kWOne:  32 sources per column as 16-bit lists src16[slot][column], one weight wc for the whole
//           layer (only with the equal-value kernels);
//   kWEdge: 32 sources per column as 16-bit lists src16[slot][column] and each edge's weight in
//           w32[slot][column] (6 bytes per edge).
constexpr int kWEll = 0, kWOne = 1, kWEdge = 2;

// Stage the 16-bit sources (and, for kWEdge, the weights) of outputs [c0, c0 + nout) of a layer
// into LDS as srcs[slot][CH] and wts[slot][CH], with 16-byte loads where the rows are aligned;
// outputs past nout get source 0 and weight 0 (they are computed but never stored).
template <int WM, int CH>
__device__ __forceinline__ void stage_lists(unsigned short *srcs, float *wts, const unsigned short *__restrict__ src16,
                                            const float *__restrict__ w32, int ncols, int c0, int nout) {
  static_assert(CH % 8 == 0, "whole 16-byte groups");
  for (int i = threadIdx.x; i < 32 * CH / 8; i += blockDim.x) {
    const int sl = i / (CH / 8), pr = (i % (CH / 8)) * 8;
    const unsigned short *sp = src16 + (size_t)sl * ncols + c0 + pr;
    uint4 v;
    if (pr + 7 < nout && (reinterpret_cast<uintptr_t>(sp) & 15) == 0) {
      v = *reinterpret_cast<const uint4 *>(sp);
    } else {
      unsigned o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int c = 0; c < 8; ++c) o[c >> 1] |= (pr + c < nout ? (unsigned)sp[c] : 0u) << (16 * (c & 1));
      v = make_uint4(o[0], o[1], o[2], o[3]);
    }
    *reinterpret_cast<uint4 *>(srcs + sl * CH + pr) = v;
  }
  if constexpr (WM == kWEdge) {
    for (int i = threadIdx.x; i < 32 * CH / 4; i += blockDim.x) {
      const int sl = i / (CH / 4), pr = (i % (CH / 4)) * 4;
      const float *wp = w32 + (size_t)sl * ncols + c0 + pr;
      float4 v;
      if (pr + 3 < nout && (reinterpret_cast<uintptr_t>(wp) & 15) == 0) {
        v = *reinterpret_cast<const float4 *>(wp);
      } else {
        v = make_float4(pr < nout ? wp[0] : 0.0f, pr + 1 < nout ? wp[1] : 0.0f, pr + 2 < nout ? wp[2] : 0.0f,
                        pr + 3 < nout ? wp[3] : 0.0f);
      }
      *reinterpret_cast<float4 *>(wts + sl * CH + pr) = v;
    }
  }
}

// Work split of one round of a layer on global tiles, tpx tiles per XCD (workgroup x runs on XCD
// x % 8; gridDim.x / 8 must be a multiple of tpx). ntl: tiles left from the round's first tile.
// With more than 8 tiles in the round, XCD x takes its tiles x, x + 8, ..., x + 8 (tpx - 1), one per
// group of its workgroups, each tile's chunks spread over the group; with at most 8 (always for
// tpx = 1), group 0 alone works and each tile's chunks are split over 8 / nt XCDs.
struct RoundSplit {
  int t;             // tile, relative to the round's first
  bool active;
  int cbeg, cend;    // the tile's chunks this XCD (part) covers
  int first, step;   // this workgroup's first chunk and stride
};
__device__ __forceinline__ RoundSplit round_split(int ntl, int tpx, int nchunks) {
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, per_xcd = gridDim.x >> 3;
  const int g = slot % tpx, per_group = per_xcd / tpx;
  const int nt = min(8 * tpx, ntl);
  RoundSplit r;
  if (nt > 8) {
    r.t = xcd + 8 * g;
    r.active = r.t < nt;
    r.cbeg = 0;
  } else {
    const int parts = nt > 0 ? 8 / nt : 1;
    r.t = xcd / parts;
    r.active = nt > 0 && g == 0 && xcd < nt * parts;
    r.cbeg = (xcd % parts) * ((nchunks + parts - 1) / parts);
    r.cend = min(nchunks, r.cbeg + (nchunks + parts - 1) / parts);
  }
  if (nt > 8) r.cend = nchunks;
  if (!r.active) r.cend = 0;
  r.first = r.cbeg + slot / tpx;
  r.step = per_group;
  return r;
}

// One round of a layer on global feature-major tiles of FMR = 32 rows: input tiles fin[t][k][b]
// (source k of list position 32t + b), output tiles fout in the same layout and positions; tiles
// [tile0, tile0 + 8) of the list, one per XCD. blockDim 256 (4 waves); a work item is a chunk of
// kGfmOutputs = 64 outputs. Lane = (row b = lane % 32, h = lane / 32): a source segment of 128
// bytes is read by 32 lanes with 4-byte loads (on gfx950 4-byte lane loads gather a segment three
// times faster than 16-byte ones), so a wave instruction serves 2 outputs; each lane runs the
// chains of the 8 consecutive outputs 16 wave + 8 h .. + 7, one slot ahead, and the results go out
// as 128-byte row segments. gridDim must be a multiple of 8: workgroup x runs on XCD x % 8, and the
// workgroups of XCD x share the output chunks of one tile, which therefore stays in that XCD's L2
// (or, for the widest layers, in the Infinity Cache) for the whole launch. With fewer than 8 tiles
// left, each tile's chunks are split over 8 / ntiles XCDs. With 16-bit lists (WM != kWEll) the
// chunk's sources (and kWEdge weights) are staged in LDS, so the gathers are the only per-output
// memory reads. Slots past the list's end hold zeros in fin and get zeros in fout.
//
// Workgroup 0 of the first round also does the list bookkeeping of the layer sequence: with
// count_out set (a layer that follows one without compaction) it counts the previous layer's live
// rows (masks_prev, complete since that kernel ended) into *count_out, and with masks_clear set it
// clears that buffer, the one the next layer will use (three buffers rotate by layer). With
// count_out set and no live row left (rows that die stay dead), the layer writes nothing.
// Live rows go to masks, or with spread set to the spread words of each tile (see or_mask). With
// cols set (kWOne only), the launch computes the ncols columns cols[p] alone, their source lists in
// src16 as [K][ncols]; the other columns equal one of these and are neither computed nor stored.
template <int WM>
__global__ __launch_bounds__(256) void k_layer_gfm(const float *__restrict__ fin, float *__restrict__ fout, int N,
                                                   const int2 *__restrict__ ell, int K,
                                                   const unsigned short *__restrict__ src16,
                                                   const float *__restrict__ w32, float wc,
                                                   const float *__restrict__ bias, float ymax,
                                                   const int *__restrict__ npos, unsigned *__restrict__ masks,
                                                   int tile0, const unsigned *__restrict__ masks_prev,
                                                   unsigned *__restrict__ masks_clear, int *__restrict__ count_out,
                                                   unsigned *__restrict__ spread, const int *__restrict__ cols,
                                                   int ncols, int tpx) {
  constexpr int FMR = 32, CH = kGfmOutputs, OPL = 8;
  static_assert(CH == 4 * 2 * OPL, "4 waves x 2 halves x OPL outputs");
  constexpr bool LISTS = WM != kWEll;
  __shared__ __align__(16) unsigned short srcs[LISTS ? 32 * CH : 8];
  __shared__ __align__(16) float wts[WM == kWEdge ? 32 * CH : 4];
  __shared__ float bstage[CH];
  __shared__ int cstage[CH];  // output column of each chunk position
  __shared__ unsigned rowmask;
  __shared__ int prev_live;
  const int R = *npos;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 64) {
    const int ntl = (R + FMR - 1) / FMR;
    int c = 0;
    if (count_out || (masks_clear && blockIdx.x == 0))
      for (int i = tid; i < ntl; i += 64) {
        if (count_out) c += __popc(masks_prev[i]);
        if (masks_clear && blockIdx.x == 0) masks_clear[i] = 0u;
      }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) c += __shfl_xor(c, d, 64);
    if (tid == 0) {
      if (count_out && blockIdx.x == 0) *count_out = c;
      prev_live = count_out ? c : 1;
      rowmask = 0u;
    }
  }
  __syncthreads();
  const int nchunks = (ncols + CH - 1) / CH;
  const RoundSplit rs = round_split((R + FMR - 1) / FMR - tile0, tpx, nchunks);
  const bool active = rs.active && prev_live != 0;  // uniform over the workgroup
  const int t = tile0 + rs.t;
  const int cend = active ? rs.cend : 0;
  const int b = lane & 31, h = lane >> 5;
  const int nvalid = active ? min(FMR, R - t * FMR) : 0;
  const float *tb = fin + (size_t)t * N * FMR + b;
  float *ob = fout + (size_t)t * N * FMR + b;
  const int jl0 = wave * 2 * OPL + h * OPL;  // this lane's outputs in the chunk: jl0 .. jl0 + OPL - 1
  bool live = false;
  for (int chunk = rs.first; chunk < cend; chunk += rs.step) {
    const int c0 = chunk * CH;
    const int nout = min(CH, ncols - c0);
    __syncthreads();  // the previous chunk is done with srcs / wts / bstage / cstage
    for (int i = tid; i < CH; i += blockDim.x) {
      const int col = i < nout ? (cols ? cols[c0 + i] : c0 + i) : 0;
      cstage[i] = col;
      bstage[i] = i < nout ? bias[col] : 0.0f;
    }
    if constexpr (LISTS) stage_lists<WM, CH>(srcs, wts, src16, w32, ncols, c0, nout);
    __syncthreads();
    float acc[OPL];
#pragma unroll
    for (int i = 0; i < OPL; ++i) acc[i] = 0.0f;
    if constexpr (LISTS) {
      // software pipeline kDepth slots deep: a slot's gathers are issued kDepth - 1 slots before
      // its fmas (each gather is one row of one output, so the depth is what keeps enough
      // segments in flight to cover the L2 latency)
      constexpr int kDepth = 4;
      float g[kDepth][OPL];
      auto fetch = [&](int sl, int bf) {
        const unsigned short *sp = srcs + sl * CH + jl0;
#pragma unroll
        for (int i = 0; i < OPL; ++i) g[bf][i] = tb[(unsigned)sp[i] * (unsigned)FMR];
      };
#pragma unroll
      for (int sl = 0; sl < kDepth - 1; ++sl) fetch(sl, sl);
#pragma unroll
      for (int sl = 0; sl < 32; ++sl) {
        if (sl + kDepth - 1 < 32) fetch(sl + kDepth - 1, (sl + kDepth - 1) % kDepth);
        // the slot's weights from LDS (two 16-byte reads), while its gathers are in flight
        float wv[OPL];
        if constexpr (WM == kWEdge) {
          const float4 x = *reinterpret_cast<const float4 *>(wts + sl * CH + jl0);
          const float4 y = *reinterpret_cast<const float4 *>(wts + sl * CH + jl0 + 4);
          wv[0] = x.x; wv[1] = x.y; wv[2] = x.z; wv[3] = x.w;
          wv[4] = y.x; wv[5] = y.y; wv[6] = y.z; wv[7] = y.w;
        } else {
#pragma unroll
          for (int i = 0; i < OPL; ++i) wv[i] = wc;
        }
        mem_fence_compiler();
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < OPL; ++i) acc[i] = fmaf(g[sl % kDepth][i], wv[i], acc[i]);
#pragma unroll
        for (int i = 0; i < OPL; i += 4) pin4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
      }
    } else {
      for (int sl = 0; sl < K; ++sl) {
#pragma unroll
        for (int i = 0; i < OPL; ++i) {
          const int2 e = ell[(size_t)sl * N + min(c0 + jl0 + i, N - 1)];
          acc[i] = fmaf(tb[(unsigned)e.x >> 2], __int_as_float(e.y), acc[i]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < OPL; ++i) {
      const int jl = jl0 + i;
      if (jl < nout) {
        const float y = activate(acc[i], bstage[jl], ymax);
        __builtin_nontemporal_store(y, ob + (size_t)cstage[jl] * FMR);
        live |= y > 0.0f;
      }
    }
  }
  // rows of this tile that stayed live in any of this workgroup's chunks: lanes b and b + 32 are
  // row b
  const unsigned long long bl = __ballot(live);
  const unsigned lm = (unsigned)bl | (unsigned)(bl >> 32);
  __syncthreads();
  if (lane == 0 && lm) atomicOr(&rowmask, lm);
  __syncthreads();
  if (tid == 0) {
    const unsigned valid = nvalid >= 32 ? 0xffffffffu : ((1u << nvalid) - 1u);  // 0 when inactive
    if (active && (rowmask & valid)) or_mask(masks, spread, t, rowmask & valid);
  }
}

// Progress word of few-tile layers, stored by workgroup 0 of each launch into coherent host memory:
// run generation (16 bits) | layer of the launch (20 bits) | live count of the previous layer (28
// bits; all ones when this launch did not count it). The host reads it to follow the device
// without copies or events, and to stop enqueuing layers once no row is live.
constexpr int kProgLayerShift = 28, kProgGenShift = 48;
constexpr unsigned long long kProgCountMask = (1ull << kProgLayerShift) - 1;
constexpr int kProgressAhead = 6;  // layers the host may enqueue ahead of the last reported one

// Partial liveness words of a few-tile layer: worker workgroup (t, s) of a launch with S slots per
// tile writes the rows of tile t that stayed live in its chunks to part[t * S + s], a plain store
// (zero or not). The tile's mask word is the OR of its S slots. Hundreds of workgroups that finish
// together would otherwise serialize on one atomic word (several us per launch).
constexpr int kPartThreads = 256;
constexpr int kPartLoads = 16;  // words per thread: kPartThreads x kPartLoads >= any launch's slots
constexpr int kMaxPartWords = kPartThreads * kPartLoads;

// Mask words m[t] = OR of the partial words of tile t (t < nt, S slots each), from the kPartLoads
// words each thread of a kPartThreads workgroup loaded (word tid + kPartThreads k). Every thread of
// the workgroup calls it; m: nt <= 8 words of LDS, returned after a barrier.
__device__ void or_partials(const unsigned (&pp)[kPartLoads], int S, int nt, unsigned *m) {
  const int tid = threadIdx.x, lane = tid & 63;
  if (tid < 8) m[tid] = 0u;
  __syncthreads();
  for (int t = 0; t < nt; ++t) {
    unsigned v = 0u;
#pragma unroll
    for (int k = 0; k < kPartLoads; ++k) v |= (tid + kPartThreads * k) / S == t ? pp[k] : 0u;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v |= __shfl_xor(v, d, 64);
    if (lane == 0 && v) atomicOr(&m[t], v);
  }
  __syncthreads();
}

__device__ __forceinline__ void load_partials(unsigned (&pp)[kPartLoads], const unsigned *part, int words) {
#pragma unroll
  for (int k = 0; k < kPartLoads; ++k) {
    const int i = threadIdx.x + kPartThreads * k;
    pp[k] = i < words ? part[i] : 0u;
  }
}

// The mask words of a few-tile layer from its partial words (before a compaction reads them).
__global__ __launch_bounds__(kPartThreads) void k_finalize_masks(const unsigned *__restrict__ part, int S, int nt,
                                                                 unsigned *__restrict__ masks) {
  __shared__ unsigned m[8];
  unsigned pp[kPartLoads];
  load_partials(pp, part, S * nt);
  or_partials(pp, S, nt, m);
  if (threadIdx.x < nt) masks[threadIdx.x] = m[threadIdx.x];
}

// Layers of few rows (at most 8 tiles, so each XCD works on one tile's share of outputs): the tile
// layout and lane mapping of k_layer_gfm with one output per lane and a whole chain's loads in
// flight at once: the KC ELL entries straight from memory (the 8 lanes of an output read the same
// entry), then all KC gathers, then the fma chain. A work item is a chunk of 32 outputs.
// Such a layer is short, so its time is mostly the latency of dependent loads. The work split
// follows ntiles_h, the host's bound on the tiles, so a lane issues its ELL loads and gathers before
// it has read the list length, which only masks the liveness bits. live_before is the live count two
// layers back (final when the launch starts); at zero every input is zero and the layer neither
// gathers nor stores. Liveness goes to partial words part_out (S = per-XCD workgroups x parts slots
// per tile). Workgroup 0 turns the previous layer's partial words part_prev (prev_S slots, prev_nt
// tiles) into its mask words masks_prev, or, with part_prev null, reads those words; then it writes
// their live count to count_out (if set) and to the progress word (if set), and clears masks_clear.
// WM picks the weight layout (kWEll, kWOne, kWEdge; see k_layer_gfm). With cols set (kWOne only),
// only the ncols columns cols[p] are computed (see k_layer_gfm).
template <int KC, int WM>
__global__ __launch_bounds__(kPartThreads) void k_layer_gfm_small(
    const float *__restrict__ fin, float *__restrict__ fout, int N, const int2 *__restrict__ ell,
    const unsigned short *__restrict__ src16, const float *__restrict__ w32, float wc,
    const float *__restrict__ bias, float ymax,
    const int *__restrict__ npos, int ntiles_h, unsigned *__restrict__ part_out,
    const unsigned *__restrict__ part_prev, int prev_S, int prev_nt, unsigned *__restrict__ masks_prev,
    unsigned *__restrict__ masks_clear, int *__restrict__ count_out, const int *__restrict__ live_before,
    unsigned long long *__restrict__ progress, unsigned long long progress_tag, const int *__restrict__ cols,
    int ncols) {
  constexpr int FMR = 32, CH = 32;
  __shared__ unsigned wmask[4];
  __shared__ unsigned pmask[8];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int parts = 8 / ntiles_h;
  const int xcd = blockIdx.x & 7;
  const int nchunks = (ncols + CH - 1) / CH;
  const int cpp = (nchunks + parts - 1) / parts;
  const int t = xcd / parts;
  const bool worker = xcd < ntiles_h * parts;
  const int cbeg = (xcd % parts) * cpp, cend = worker ? min(nchunks, cbeg + cpp) : 0;
  const int q = lane & 7, h = lane >> 3;
  const int per_xcd = gridDim.x >> 3;
  const char *tbase = reinterpret_cast<const char *>(fin + (size_t)t * N * FMR) + q * 16;
  float *obase = fout + (size_t)t * N * FMR + q * 4;
  const bool wg0 = blockIdx.x == 0;
  // no row was live two layers back: every input is zero, so the layer gathers nothing and stores
  // nothing, and its rows stay dead. The count is read through a per-lane (zero) offset, which keeps
  // it a vector value: used as a scalar it would be waited for before the ELL loads are issued.
  int zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
  const int count_before = __hip_atomic_load(live_before + zero, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // workgroup 0: the previous layer's partial words, in flight during its chunk
  unsigned pp[kPartLoads];
  if (wg0 && part_prev) load_partials(pp, part_prev, prev_S * prev_nt);
  int R = 0;           // list length
  unsigned pm = 0u;    // lane i < ntiles_h of workgroup 0: the previous layer's mask word of tile i
  unsigned lm = 0u;
  // FIRST: the workgroup's first chunk, which also issues the loads of the list length and the
  // previous masks
  auto run_chunk = [&](int chunk, auto first) {
    constexpr bool FIRST = decltype(first)::value;
    const int j = chunk * CH + wave * 8 + h;
    const int jj = min(j, ncols - 1);
    const int col = cols ? cols[jj] : jj;  // output column
    // byte offsets of the sources' segments and the weights (16-bit source lists with one weight wc
    // or each edge's weight beside them, or ELL entries)
    unsigned eo[KC];
    float ew[KC];
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      if constexpr (WM != kWEll) {
        eo[i] = (unsigned)src16[(size_t)i * ncols + jj] * (FMR * 4);
        ew[i] = WM == kWEdge ? w32[(size_t)i * ncols + jj] : wc;
      } else {
        const int2 e = ell[(size_t)i * N + jj];
        eo[i] = (unsigned)e.x;
        ew[i] = __int_as_float(e.y);
      }
    }
    const float b = bias[col];
    // taken here, after the ELL loads (the asm keeps the compare from being hoisted above them)
    int cb = count_before;
    asm volatile("" : "+v"(cb));
    const bool dead = cb == 0;
#pragma unroll
    for (int i = 0; i < KC; ++i) eo[i] = dead ? 0u : eo[i];
    float4 g[KC];
#pragma unroll
    for (int i = 0; i < KC; ++i) g[i] = *reinterpret_cast<const float4 *>(tbase + eo[i]);
    if constexpr (FIRST) {
      // after the gathers: vector loads complete in order, so waiting for these waits for nothing
      // the fma chain does not need anyway
      R = __hip_atomic_load(npos, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (wg0 && !part_prev && count_out)
        pm = __hip_atomic_load(masks_prev + min(lane, ntiles_h - 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // every gather is issued before the first fma waits on one
    mem_fence_compiler();
    __builtin_amdgcn_sched_barrier(0);
    float a[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      const float w = ew[i];
      a[0] = fmaf(g[i].x, w, a[0]);
      a[1] = fmaf(g[i].y, w, a[1]);
      a[2] = fmaf(g[i].z, w, a[2]);
      a[3] = fmaf(g[i].w, w, a[3]);
    }
    // the chain is computed for every lane (outputs past N repeat output N - 1), so the loads stay
    // ahead of the branch that stores
    const float4 y = make_float4(activate(a[0], b, ymax), activate(a[1], b, ymax), activate(a[2], b, ymax),
                                 activate(a[3], b, ymax));
    const unsigned bits = (y.x > 0.0f ? 1u : 0u) | (y.y > 0.0f ? 2u : 0u) | (y.z > 0.0f ? 4u : 0u) | (y.w > 0.0f ? 8u : 0u);
    lm |= (j < ncols ? bits : 0u) << (4 * q);
    // positions past the list length (up to the host's tile bound) are stored too: nothing reads them
    if (j < ncols && !dead) store_stream(reinterpret_cast<float4 *>(obase + (size_t)col * FMR), y);
  };
  int chunk = cbeg + (int)(blockIdx.x >> 3);
  if (chunk < cend) {
    run_chunk(chunk, std::true_type{});
    for (chunk += per_xcd; chunk < cend; chunk += per_xcd) run_chunk(chunk, std::false_type{});
  }
  if (wg0) {
    // (workgroup 0 always runs chunk 0, so R is loaded)
    const int ntiles = min(8, (R + FMR - 1) / FMR);
    if (part_prev) {
      or_partials(pp, prev_S, prev_nt, pmask);
      if (tid < prev_nt) masks_prev[tid] = pmask[tid];
      pm = lane < prev_nt ? pmask[lane] : 0u;
    }
    if (wave == 0) {
      int c = __popc(lane < ntiles ? pm : 0u);
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) c += __shfl_xor(c, d, 64);
      if (lane == 0 && count_out) *count_out = c;
      if (lane == 0 && progress)
        __hip_atomic_store(progress, progress_tag | (count_out ? (unsigned long long)c : kProgCountMask),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      if (masks_clear && lane < ntiles) masks_clear[lane] = 0u;
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) lm |= __shfl_xor(lm, d, 64);
  if (lane == 0) wmask[wave] = lm;
  __syncthreads();
  if (tid == 0 && worker) {
    const int nvalid = min(FMR, R - t * FMR);
    const unsigned valid = nvalid >= 32 ? 0xffffffffu : (nvalid > 0 ? (1u << nvalid) - 1u : 0u);
    const int S = per_xcd * parts;
    part_out[t * S + (blockIdx.x >> 3) * parts + xcd % parts] =
        count_before == 0 ? 0u : (wmask[0] | wmask[1] | wmask[2] | wmask[3]) & valid;
  }
}

constexpr int kBitsThreads = 1024;  // k_layer_bits workgroup: 16 waves, up to 128 registers each
// k_layer_bits' table that turns 4 input bits into 4 floats: 16 entries of 16 bytes (a 256-entry
// table of 8 bits measured twice as slow: its reads spread over more banks)
constexpr int kLutF4 = 16;
// k_layer_bits' LDS tile: one bit word per neuron, sized for the widest network of its height
// (T = 32 for up to 16384 neurons, 16 for up to 65536); static, so that its address is a constant
// that folds into the LDS instructions' offsets. Beside it: the table, the mask word and the
// dictionary cache (under 9 KiB).
__host__ __device__ constexpr int bits_tile_bytes(int T) { return T == 32 ? 16384 * 4 : 65536 * 2; }
static_assert(bits_tile_bytes(16) + 9 * 1024 <= 160 * 1024, "LDS of k_layer_bits");

// Value dictionary for one-byte activation codes, in device memory (kDictWords words):
//   val[256]   the value (fp32 bit pattern) of each code: decoding is val[code];
//   key[1024]  an open-addressing hash table of the values seen, by dict_hash (four slots per code,
//              so that probes stay short also when the 256 codes run out);
//   code[1024] the code of the value in each hash slot (kNoCode until it is published);
//   next       the next free code.
// Codes are handed out in order 0, 1, 2, ... (code 0 is +0.0, whose key sits in its hash slot 0
// from the start), so a layer's first 32 values decode from distinct LDS banks. A value's slot is
// claimed with compare-and-swap; the lane that claims it takes the next code and publishes it
// (relaxed device-scope atomics: a reader needs the code word itself, and the values are read by
// later kernels only); slots and codes never change afterwards, so a workgroup may cache them in
// LDS. kDictEmpty (a
// NaN pattern, never an activation) marks free slots.
// a value whose slot was claimed by another lane waits this many reads at most for its code (the
// claimer publishes it a few instructions after its compare-and-swap); past the bound the
// dictionary counts as full, which sends the layer to its fp32 outputs
constexpr int kDictWaitReads = 1 << 16;
// Code tiles hold CR list positions (code_rows below): [tile][N][CR] bytes, list position p at tile
// p / CR, byte p % CR.
// The code-tile height goes with the bit tiles that write them: 128 rows after 32-row bit tiles,
// whose counting workgroups then fill each 128-byte segment in 4 parts; 64 rows after 16-row bit
// tiles (4 parts each as well). Taller segments serve more rows per gather request.
__host__ __device__ constexpr int code_rows(int T) { return T == 32 ? 128 : 64; }
// rows per lane of k_layer_gfm_u8 (8: 8-byte gathers, for 64-row codes; 4 for 128-row codes, whose
// lanes would otherwise hold too many accumulators)
#ifndef SDNN_U8_RPL
#define SDNN_U8_RPL 8
#endif
__host__ __device__ constexpr int u8_rows_per_lane(int CR) { return CR == 64 ? SDNN_U8_RPL : 4; }
// outputs per lane of k_layer_gfm_u8 (at most 32 / rows per lane accumulators' worth)
#ifndef SDNN_U8_OPL
#define SDNN_U8_OPL (32 / SDNN_U8_RPL)
#endif
__host__ __device__ constexpr int u8_outs_per_lane(int CR) { return CR == 64 ? SDNN_U8_OPL : 8; }
// outputs per work item: 4 waves x outputs per wave instruction (64 / lanes per code segment) x
// outputs per lane
__host__ __device__ constexpr int u8_outputs(int CR) {
  return 4 * (64 / (CR / u8_rows_per_lane(CR))) * u8_outs_per_lane(CR);
}
// k_layer_gfm_u8's software pipeline: slots whose gathers are in flight (SDNN_U8_DEPTH - 1 ahead),
// code dwords whose dictionary reads run ahead of the fmas (SDNN_U8_LA), waves per SIMD the
// registers are held to at 64-row codes (SDNN_U8_WAVES)
#ifndef SDNN_U8_DEPTH
#define SDNN_U8_DEPTH 2
#endif
#ifndef SDNN_U8_LA
#define SDNN_U8_LA 2
#endif
#ifndef SDNN_U8_WAVES
#define SDNN_U8_WAVES 5
#endif
// One XCD's L2. Two-byte codes are tried only for layers whose fp32 input tile (32 rows of every
// source) is larger: at 65536 sources they gather faster than the fp32 tiles, which live in the
// Infinity Cache, while at 16384 the fp32 tiles stay in L2 and the codes (whose 4096-entry
// dictionary also halves the workgroups per CU) measure slower, encoding included.
constexpr size_t kXcdL2Bytes = (size_t)4 << 20;

template <int CB = 1>
__device__ __forceinline__ unsigned dict_hash(unsigned key) {
  // (low 24 bits of key ^ (key >> 16)) * 0x9E3779, bits kHashShift.. (full-rate 24-bit multiply);
  // key 0 hashes to slot 0
  unsigned h;
  asm("v_mul_u32_u24 %0, 0x9e3779, %1" : "=v"(h) : "v"(key ^ (key >> 16)));
  return (h >> DictShape<CB>::kHashShift) & (unsigned)(DictShape<CB>::kHash - 1);
}

// A workgroup's LDS cache of the dictionary: kCacheEntries (key, code) entries in two-way sets
// (entries 2i and 2i + 1), set chosen by a multiplicative hash (a 24-bit multiply, full rate) that
// spreads the values of a layer well (checked on the workloads' value sets). An entry is claimed
// once, by compare-and-swap of its key from kDictEmpty to kCacheBusy; the claimer writes the code,
// then the key (one wave's LDS operations take effect in order; a compiler barrier keeps the order);
// entries are never replaced. A reader loads the keys before the codes, so a key it sees has its
// code in place; kCacheBusy (a NaN pattern) never matches a value.
constexpr int kCacheEntries = DictShape<1>::kCache;
constexpr unsigned kCacheBusy = 0x7fc00001u;
template <int CB = 1>
__device__ __forceinline__ unsigned cache_set(unsigned key) {  // first entry of the key's set (even)
  // the low 32 bits of (low 24 bits of key ^ (key >> 16)) times 0x9E3779, by the full-rate 24-bit
  // multiply (the compiler would pick the quarter-rate 32-bit one)
  unsigned h;
  asm("v_mul_u32_u24 %0, 0x9e3779, %1" : "=v"(h) : "v"(key ^ (key >> 16)));
  return (h >> DictShape<CB>::kCacheShift) & (unsigned)(DictShape<CB>::kCache - 2);
}

// Code of the value with bits `key` from the global table, claiming a free slot and a code on the
// way, then recorded in the LDS cache (dlk, dlc) if its set has a free entry. A full dictionary
// sets *overflow and returns 0; the caller's output is then not used. Once *overflow is set (by any
// lane) every call returns at its next probe.
template <int CB = 1>
__device__ __forceinline__ unsigned dict_code_slow(unsigned key, unsigned *dlk, unsigned *dlc, unsigned *gd,
                                                   int *overflow) {
  constexpr int SLOTS = DictShape<CB>::kSlots, HASH = DictShape<CB>::kHash;
  unsigned *gkey = gd + dict_key_off<CB>(), *gcode = gd + dict_code_off<CB>();
  unsigned h = dict_hash<CB>(key);
  for (int i = 0; i < HASH; ++i) {
    if (__hip_atomic_load(overflow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return 0;
    unsigned cur = __hip_atomic_load(&gkey[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool won = false;
    if (cur == kDictEmpty) {
      const unsigned prev = atomicCAS(&gkey[h], kDictEmpty, key);
      won = prev == kDictEmpty;
      cur = won ? key : prev;
    }
    if (won) {
      // this lane claimed the slot: it takes the next code, records the value, publishes the code
      const unsigned c = atomicAdd(gd + dict_next_off<CB>(), 1u);
      if (c < (unsigned)SLOTS) gd[c] = key;
      __hip_atomic_store(&gcode[h], c < (unsigned)SLOTS ? c : kNoCode - 1u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    if (cur == key) {
      unsigned c = kNoCode;
      for (int it = 0; it < kDictWaitReads && c == kNoCode; ++it)
        c = __hip_atomic_load(&gcode[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (c >= (unsigned)SLOTS) break;  // no code left, or none published within the bound
      const unsigned st = cache_set<CB>(key);
      if (dlk[st] != key && dlk[st + 1] != key) {
#pragma unroll
        for (unsigned wy = 0; wy < 2; ++wy) {
          if (atomicCAS(&dlk[st + wy], kDictEmpty, kCacheBusy) == kDictEmpty) {
            dlc[st + wy] = c;
            mem_fence_compiler();
            __hip_atomic_store(&dlk[st + wy], key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            break;
          }
        }
      }
      return c;
    }
    h = (h + 1) & (HASH - 1);
  }
  *overflow = 1;
  return 0;
}
// The cache's answer for `key`: *code, and whether it was there.
template <int CB = 1>
__device__ __forceinline__ bool cache_lookup(unsigned key, const unsigned *dlk, const unsigned *dlc, unsigned *code) {
  const unsigned st = cache_set<CB>(key);
  const uint2 k = *reinterpret_cast<const uint2 *>(dlk + st);
  mem_fence_compiler();  // the keys are read before the codes
  const uint2 c = *reinterpret_cast<const uint2 *>(dlc + st);
  *code = k.x == key ? c.x : c.y;
  return k.x == key || k.y == key;
}
template <int CB = 1>
__device__ __forceinline__ unsigned dict_code(float y, unsigned *dlk, unsigned *dlc, unsigned *gd, int *overflow) {
  const unsigned key = __float_as_uint(y);
  unsigned c;
  if (cache_lookup<CB>(key, dlk, dlc, &c)) return c;
  return dict_code_slow<CB>(key, dlk, dlc, gd, overflow);
}

// waves per SIMD the registers of k_layer_gfm_u8 are held to (with two-byte codes and staged weights,
// 40 KiB of LDS per workgroup leave room for 3)
constexpr int u8_waves(int WM, int CR, int CB) {
  return CB == 2 && WM == kWEdge ? 3 : CR == 64 && CB == 1 ? SDNN_U8_WAVES : 4;
}

// One round of a layer whose input tiles hold CB-byte codes of the activations, cin[t][k][b]
// (source k of list position CR t + b), decoded as dict[code]; the output is fp32 tiles of 32 rows
// as in k_layer_gfm (code tile t covers output tiles ST t .. ST t + ST - 1, ST = CR / 32). Code tiles
// [tile0, tile0 + 8) go one per XCD, as in k_layer_gfm. Two-byte codes (CB = 2, 4096-entry
// dictionary, CR = 64) double the bytes of every gather and leave the rest as it is. A code segment
// is CR codes: RL = CR / RPL lanes read it, RPL codes each (RPL = 4: 4-byte loads; 8: 8-byte loads,
// which halves the gather instructions and their address arithmetic; 16-byte loads for two-byte
// codes), so a wave instruction serves OPI = 64 / RL outputs.
// Lane = (r = lane % RL: rows RPL r .. RPL r + RPL - 1, o = lane / RL); the lane runs the OPL
// consecutive outputs jw + OPL o .. + OPL - 1 of its wave's block of OPI * OPL (4 OPL RPL = 128
// accumulator rows per lane would not fit: OPL RPL = 32), so for every slot its sources come from
// LDS one 16-bit read each and its weights in 16-byte reads. A work item is a chunk of 4 waves'
// outputs. The dictionary and the chunk's lists sit in LDS (kWEdge: 6 bytes per entry, 24 KiB,
// which leaves room for 5 workgroups per CU; 40 KiB with the two-byte codes' dictionary). A 32-row
// output segment that is zero in every row is not stored; its bit in seglive (one bit per fp32
// tile and source) says so. Registers are held to 5 waves per SIMD for one-byte 64-row codes (more
// waves keep more gathers in flight; 6 spill), 4 for 128-row codes and 3 for two-byte codes with
// staged weights (u8_waves). Live rows go to masks, or with spread set to the spread words of each
// fp32 tile (see or_mask). With cols set (kWOne only), the launch computes the ncols columns
// cols[p] alone (see k_layer_gfm), stores every segment of them and leaves seglive untouched.
template <int WM, int CR, int RPL, int OPL, int CB = 1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(u8_waves(WM, CR, CB)))) void k_layer_gfm_u8(
    const unsigned char *__restrict__ cin, float *__restrict__ fout, int N, const int2 *__restrict__ ell, int K,
    const unsigned short *__restrict__ src16, const float *__restrict__ w32, float wc, const float *__restrict__ bias,
    float ymax, const float *__restrict__ dict, const int *__restrict__ npos, unsigned *__restrict__ masks,
    unsigned *__restrict__ seglive, int tile0, unsigned *__restrict__ spread, const int *__restrict__ cols, int ncols,
    int tpx) {
  static_assert(RPL == 4 || RPL == 8, "4 or 8 rows per lane");
  static_assert(OPL == 2 || OPL % 4 == 0, "weights are read in pairs or quads");
  static_assert(OPL * RPL <= 32, "accumulators per lane");
  constexpr int RL = CR / RPL, OPI = 64 / RL, CH = 4 * OPI * OPL, ST = CR / 32;
  constexpr int DW = RPL * CB / 4;  // code dwords per gather
  constexpr int CPD = 4 / CB;       // codes per dword
  constexpr unsigned CMASK = (unsigned)DictShape<CB>::kSlots - 1u;  // (codes below kSlots)
  constexpr int LPS = 32 / RPL;     // lanes per 32-row output segment
  static_assert(CB == 1 || CB == 2, "one- or two-byte codes");
  constexpr bool LISTS = WM != kWEll;
  static_assert(CR == 64 || CR == 128, "code segments of 64 or 128 rows");
  static_assert(CH % 32 == 0 && CH == u8_outputs(CR), "a chunk covers whole bitmap words");
  static_assert(32 % (OPI * OPL) == 0 || (OPI * OPL) % 32 == 0, "bitmap words");
  static_assert(OPI * OPL <= 32, "a wave's outputs lie within one bitmap word");
  __shared__ float dl[DictShape<CB>::kSlots];
  __shared__ __align__(16) unsigned short srcs[LISTS ? 32 * CH : 8];
  __shared__ __align__(16) float wts[WM == kWEdge ? 32 * CH : 4];
  __shared__ float bstage[CH];
  __shared__ int cstage[CH];  // output column of each chunk position
  __shared__ unsigned segw[ST][CH / 32];
  __shared__ unsigned long long rowmask[CR / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < DictShape<CB>::kSlots; i += blockDim.x) dl[i] = dict[i];
  if (tid < CR / 64) rowmask[tid] = 0ull;
  const int R = *npos;
  const int nchunks = (ncols + CH - 1) / CH;
  const RoundSplit rs = round_split((R + CR - 1) / CR - tile0, tpx, nchunks);
  const bool active = rs.active;
  const int t = tile0 + rs.t;
  const int cend = rs.cend;
  const int r = lane % RL, o = lane / RL;
  const int nvalid = active ? min(CR, R - t * CR) : 0;
  // output rows RPL r .. of the code tile: fp32 tile ST t + RPL r / 32, slots (RPL r) % 32; the
  // list's fp32 tiles end at (R + 31) / 32, so the last code tile may lack some of its fp32 tiles
  const int otile = ST * t + (RPL * r) / 32;
  float *obase = fout + ((size_t)otile * N) * 32 + (RPL * r) % 32;
  const bool has_tile = otile * 32 < R;
  const int NW = (N + 31) / 32;
  // the tile base is uniform, so a gather is one 32-bit offset from it
  const unsigned char *tbs = cin + (size_t)t * N * CR * CB;
  const unsigned lofs = (unsigned)(RPL * r * CB);  // byte offset of the lane's rows in a segment
  // live rows seen by this lane: bit (RPL r + c) % 64 of word (RPL r) / 64
  unsigned long long lm[CR / 64];
#pragma unroll
  for (int h = 0; h < CR / 64; ++h) lm[h] = 0ull;
  const int jw = wave * OPI * OPL;  // first output of this wave in the chunk
  const int jl0 = jw + o * OPL;     // this lane's outputs: jl0 .. jl0 + OPL - 1
  for (int chunk = rs.first; chunk < cend; chunk += rs.step) {
    const int c0 = chunk * CH;
    const int nout = min(CH, ncols - c0);
    __syncthreads();  // the previous chunk is done with srcs / wts / bstage / cstage / segw
    for (int i = tid; i < CH; i += blockDim.x) {
      const int col = i < nout ? (cols ? cols[c0 + i] : c0 + i) : 0;
      cstage[i] = col;
      bstage[i] = i < nout ? bias[col] : 0.0f;
    }
    if (tid < ST * (CH / 32)) segw[tid / (CH / 32)][tid % (CH / 32)] = 0u;
    if constexpr (LISTS) stage_lists<WM, CH>(srcs, wts, src16, w32, ncols, c0, nout);
    __syncthreads();
    float acc[OPL][RPL];
#pragma unroll
    for (int i = 0; i < OPL; ++i)
#pragma unroll
      for (int c = 0; c < RPL; ++c) acc[i][c] = 0.0f;
    if constexpr (LISTS) {
      // software pipeline: a slot's gathers are issued one slot before its fmas (deeper pipelines
      // measure no faster: the gathers are limited by the vector-memory path, not by latency)
      constexpr int kDepth = SDNN_U8_DEPTH;
      unsigned wd[kDepth][OPL][DW];
      auto fetch = [&](int sl, int bf) {
        const unsigned short *sp = srcs + sl * CH + jl0;
#pragma unroll
        for (int i = 0; i < OPL; ++i) {
          const unsigned char *gp = tbs + ((unsigned)sp[i] * (unsigned)(CR * CB) + lofs);
          if constexpr (DW == 4) {
            const uint4 v = *reinterpret_cast<const uint4 *>(gp);
            wd[bf][i][0] = v.x;
            wd[bf][i][1] = v.y;
            wd[bf][i][2] = v.z;
            wd[bf][i][3] = v.w;
          } else if constexpr (DW == 2) {
            const uint2 v = *reinterpret_cast<const uint2 *>(gp);
            wd[bf][i][0] = v.x;
            wd[bf][i][1] = v.y;
          } else {
            wd[bf][i][0] = *reinterpret_cast<const unsigned *>(gp);
          }
        }
      };
#pragma unroll
      for (int sl = 0; sl < kDepth - 1; ++sl) fetch(sl, sl);
#pragma unroll
      for (int sl = 0; sl < 32; ++sl) {
        if (sl + kDepth - 1 < 32) fetch(sl + kDepth - 1, (sl + kDepth - 1) % kDepth);
        mem_fence_compiler();
        __builtin_amdgcn_sched_barrier(0);
        // the slot's weights from LDS (16-byte reads, ahead of the dictionary reads below)
        float wv[OPL];
        if constexpr (WM == kWEdge && OPL == 2) {
          const float2 a = *reinterpret_cast<const float2 *>(wts + sl * CH + jl0);
          wv[0] = a.x; wv[1] = a.y;
        } else if constexpr (WM == kWEdge) {
#pragma unroll
          for (int i = 0; i < OPL; i += 4) {
            const float4 a = *reinterpret_cast<const float4 *>(wts + sl * CH + jl0 + i);
            wv[i] = a.x; wv[i + 1] = a.y; wv[i + 2] = a.z; wv[i + 3] = a.w;
          }
        } else {
#pragma unroll
          for (int i = 0; i < OPL; ++i) wv[i] = wc;
        }
        // dictionary lookups run LA code dwords ahead of the fmas that use them
        constexpr int NQ = OPL * DW;  // code dwords of the slot
        constexpr int LA = SDNN_U8_LA;
        float dv[LA + 1][CPD];
        auto lookup = [&](int q) {
#pragma unroll
          for (int c = 0; c < CPD; ++c)
            dv[q % (LA + 1)][c] = dl[(wd[sl % kDepth][q / DW][q % DW] >> (8 * CB * c)) & CMASK];
        };
#pragma unroll
        for (int q = 0; q < LA; ++q) lookup(q);
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          if (q + LA < NQ) lookup(q + LA);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int c = 0; c < CPD; ++c)
            acc[q / DW][CPD * (q % DW) + c] = fmaf(dv[q % (LA + 1)][c], wv[q / DW], acc[q / DW][CPD * (q % DW) + c]);
          __builtin_amdgcn_sched_barrier(0);
        }
        // this slot's fmas complete here, before the slot after next is fetched
#pragma unroll
        for (int i = 0; i < OPL; ++i)
#pragma unroll
          for (int c = 0; c < RPL; c += 4) pin4(acc[i][c], acc[i][c + 1], acc[i][c + 2], acc[i][c + 3]);
      }
    } else {
      const unsigned char *tb = tbs + lofs;
      for (int sl = 0; sl < K; ++sl) {
#pragma unroll
        for (int i = 0; i < OPL; ++i) {
          const int2 e = ell[(size_t)sl * N + min(c0 + jl0 + i, N - 1)];
#pragma unroll
          for (int d = 0; d < DW; ++d) {
            const unsigned word = *reinterpret_cast<const unsigned *>(tb + ((unsigned)e.x >> 7) * (CR * CB) + 4 * d);
#pragma unroll
            for (int c = 0; c < CPD; ++c)
              acc[i][CPD * d + c] = fmaf(dl[(word >> (8 * CB * c)) & CMASK], __int_as_float(e.y), acc[i][CPD * d + c]);
          }
        }
      }
    }
    // segment bits of this wave's outputs (jw .. jw + OPI OPL - 1, within one bitmap word), per fp32 tile
    unsigned seg[ST];
#pragma unroll
    for (int q = 0; q < ST; ++q) seg[q] = 0u;
#pragma unroll
    for (int i = 0; i < OPL; ++i) {
      const int jl = jl0 + i;
      const float b = bstage[jl];
      float y[RPL];
      unsigned bits = 0u;
#pragma unroll
      for (int c = 0; c < RPL; ++c) {
        y[c] = activate(acc[i][c], b, ymax);
        bits |= (jl < nout && y[c] > 0.0f ? 1u : 0u) << c;
      }
      const unsigned long long bal = __ballot(bits != 0u);
      // the LPS lanes of this lane's output segment: lanes (lane & ~(LPS - 1)) .. + LPS - 1
      constexpr unsigned long long kSegLanes = (1ull << LPS) - 1ull;
      if (jl < nout && has_tile && (cols || ((bal >> (lane & ~(LPS - 1))) & kSegLanes) != 0ull)) {
#pragma unroll
        for (int c = 0; c < RPL; c += 4)
          store_stream(reinterpret_cast<float4 *>(obase + (size_t)cstage[jl] * 32 + c),
                       make_float4(y[c], y[c + 1], y[c + 2], y[c + 3]));
      }
#pragma unroll
      for (int h = 0; h < CR / 64; ++h)
        if ((RPL * r) / 64 == h) lm[h] |= (unsigned long long)bits << ((RPL * r) % 64);
      // output jw + OPL oo + i of fp32 tile q is stored by lanes oo RL + LPS q .. + LPS - 1
#pragma unroll
      for (int oo = 0; oo < OPI; ++oo)
#pragma unroll
        for (int q = 0; q < ST; ++q)
          seg[q] |= (((bal >> (oo * RL + LPS * q)) & kSegLanes) != 0ull ? 1u : 0u) << ((jw % 32) + oo * OPL + i);
    }
    if (lane == 0)
#pragma unroll
      for (int q = 0; q < ST; ++q)
        if (seg[q]) atomicOr(&segw[q][jw / 32], seg[q]);
    __syncthreads();
    if (tid < ST * (CH / 32) && !cols) {
      const int q = tid / (CH / 32), wi = tid % (CH / 32);
      if ((ST * t + q) * 32 < R && c0 + 32 * wi < N) seglive[(size_t)(ST * t + q) * NW + c0 / 32 + wi] = segw[q][wi];
    }
  }
  // rows of this code tile that stayed live in any of this workgroup's chunks
#pragma unroll
  for (int h = 0; h < CR / 64; ++h)
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) lm[h] |= __shfl_xor(lm[h], d, 64);
  __syncthreads();
  if (lane == 0)
#pragma unroll
    for (int h = 0; h < CR / 64; ++h)
      if (lm[h]) atomicOr(&rowmask[h], lm[h]);
  __syncthreads();
  if (tid == 0 && active) {
#pragma unroll
    for (int q = 0; q < ST; ++q) {
      const int lo = 32 * q;  // rows lo .. lo + 31 of the code tile
      const unsigned valid = nvalid - lo >= 32 ? 0xffffffffu : (nvalid > lo ? ((1u << (nvalid - lo)) - 1u) : 0u);
      const unsigned m = (unsigned)(rowmask[q / 2] >> (32 * (q & 1))) & valid;
      if (m) or_mask(masks, spread, ST * t + q, m);
    }
  }
}

// Repack of one-byte code tiles (CR positions each) after a compaction: position p of the
// new tiles takes the code at position src[p] of the old ones; positions past *npos get code 0
// (+0.0). A thread writes 4 codes of one source.
template <int CR>
__global__ __launch_bounds__(256) void k_repack_u8(const unsigned char *__restrict__ sfm, unsigned char *__restrict__ dfm,
                                                   int N, const int *__restrict__ src, const int *__restrict__ npos) {
  constexpr int QPS = CR / 4;  // 4-byte quads per source segment
  const int R = *npos;
  const int ntiles = (R + CR - 1) / CR;
  const size_t items = (size_t)ntiles * N * QPS;
  for (size_t it = blockIdx.x * (size_t)blockDim.x + threadIdx.x; it < items; it += (size_t)gridDim.x * blockDim.x) {
    const int qd = (int)(it % QPS);
    const size_t rest = it / QPS;
    const int k = (int)(rest % N);
    const int t = (int)(rest / N);
    unsigned word = 0u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int p = t * CR + qd * 4 + c;
      if (p < R) {
        const int sp = src[p];
        word |= (unsigned)sfm[((size_t)(sp / CR) * N + k) * CR + sp % CR] << (8 * c);
      }
    }
    *reinterpret_cast<unsigned *>(dfm + ((size_t)t * N + k) * CR + qd * 4) = word;
  }
}

template <int T>
struct BitWord;
template <>
struct BitWord<16> {
  using type = unsigned short;
};
template <>
struct BitWord<32> {
  using type = unsigned int;
};

// The value dictionary back to its initial state (code 0 = +0.0, every other slot free, next code
// 1) and its overflow flag cleared, before a later layer's outputs are encoded into it.
template <int CB>
__global__ void k_dict_reset(unsigned *__restrict__ dict, int *__restrict__ overflow) {
  dict_init<CB>(dict, blockIdx.x * blockDim.x + threadIdx.x, gridDim.x * blockDim.x);
  if (blockIdx.x == 0 && threadIdx.x == 0) *overflow = 0;
}

// Encode the fp32 tiles of a layer's input (32 list positions each) as CB-byte dictionary codes in
// tiles of CR positions, cout[t][k][b] = code of the value at list position CR t + b of source k,
// so that the layer can gather them with k_layer_gfm_u8 (exact: a code decodes to the stored bits).
// A thread encodes 16 positions of one source (16 CB bytes, one or two 16-byte stores). Positions
// at or past *npos get code 0 and are not read. Codes come from gd (the dictionary of CB-byte
// codes) through a per-workgroup LDS cache, as in k_layer_bits; more distinct values than the
// dictionary holds set *overflow, and every thread stops at its next item (the caller then keeps
// the fp32 tiles).
template <int CR, int CB>
__global__ __launch_bounds__(256) void k_encode(const float *__restrict__ fin, unsigned char *__restrict__ cout, int N,
                                                const int *__restrict__ npos, unsigned *__restrict__ gd,
                                                int *__restrict__ overflow) {
  constexpr int CE = DictShape<CB>::kCache;
  __shared__ __align__(8) unsigned dlk[CE];
  __shared__ __align__(8) unsigned dlc[CE];
  for (int i = threadIdx.x; i < CE; i += blockDim.x) dlk[i] = kDictEmpty;
  __syncthreads();
  const int R = *npos;
  constexpr int QPS = CR / 16;  // 16-position groups per source segment
  const size_t items = (size_t)((R + CR - 1) / CR) * N * QPS;
  const size_t step = (size_t)gridDim.x * blockDim.x;
  for (size_t it = (size_t)blockIdx.x * blockDim.x + threadIdx.x; it < items; it += step) {
    if (__hip_atomic_load(overflow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    const int q = (int)(it % QPS);
    const size_t rest = it / QPS;
    const int k = (int)(rest % N);
    const size_t t = rest / N;
    const int p0 = (int)t * CR + q * 16;  // first list position of the group
    unsigned code[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) code[u] = 0u;
    if (p0 < R) {
      // the group lies in one 32-position fp32 tile (p0 % 16 == 0)
      const float4 *src = reinterpret_cast<const float4 *>(fin + ((size_t)(p0 >> 5) * N + k) * 32 + (p0 & 31));
      float v[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 x = src[g];
        v[4 * g] = x.x; v[4 * g + 1] = x.y; v[4 * g + 2] = x.z; v[4 * g + 3] = x.w;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = p0 + u < R ? v[u] : 0.0f;
      bool miss = false;
#pragma unroll
      for (int u = 0; u < 16; ++u) miss |= !cache_lookup<CB>(__float_as_uint(v[u]), dlk, dlc, &code[u]);
      if (miss) {
#pragma unroll
        for (int u = 0; u < 16; ++u) code[u] = dict_code<CB>(v[u], dlk, dlc, gd, overflow);
      }
    }
    uint4 *dst = reinterpret_cast<uint4 *>(cout + ((t * N + k) * CR + q * 16) * CB);
    if constexpr (CB == 1) {
      uint4 w;
      w.x = code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
      w.y = code[4] | (code[5] << 8) | (code[6] << 16) | (code[7] << 24);
      w.z = code[8] | (code[9] << 8) | (code[10] << 16) | (code[11] << 24);
      w.w = code[12] | (code[13] << 8) | (code[14] << 16) | (code[15] << 24);
      store_stream(dst, w);
    } else {
      store_stream(dst, make_uint4(code[0] | (code[1] << 16), code[2] | (code[3] << 16), code[4] | (code[5] << 16),
                                   code[6] | (code[7] << 16)));
      store_stream(dst + 1, make_uint4(code[8] | (code[9] << 16), code[10] | (code[11] << 16),
                                       code[12] | (code[13] << 16), code[14] | (code[15] << 16)));
    }
  }
}

// Reports the overflow flag to the host through the coherent report word (as k_compact does,
// with a count of 0).
__global__ void k_report_overflow(const int *__restrict__ overflow, unsigned long long *__restrict__ notify,
                                  unsigned long long tag) {
  const unsigned long long flags = *overflow != 0 ? 2ull : 0ull;
  __hip_atomic_store(notify, (tag << 40) | (flags << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// After a compaction of the global-tile path: move the live positions of a layer's output tiles
// into fresh tiles, dst[t][k][b] = the value at list position src[32t + b] of the source tiles
// (tile src / 32, slot src % 32), for positions below *npos; zero past it. A work item is one new
// tile and kRepackSources sources. The new tile's rows come from at most 32 old tiles (src is
// ascending); for each of them, 8 lanes read a source's whole 128-byte segment (one 16-byte load
// each), keep the rows the new tile takes, and place them in an LDS stage from which the new
// segments are written whole. So each needed old segment is read once, coalesced. With seglive
// set, an old segment whose bit there is clear was never stored (all its rows are zero) and is not
// read. With cols set (tiles of a layer that computed only the columns cols[0..ncols); seglive is
// then null), only those sources are moved.
// With CB = 1 the new tiles are written as one-byte dictionary codes instead, in code tiles of CR
// positions as k_encode writes them (dcodes; cols must be null): the repack and the encoding of the
// next layer's inputs in one pass. Every position of the last code tile is written (code 0 past
// *npos). A full dictionary sets *overflow, and the workgroups stop at their next work item (the
// caller then repacks the fp32 tiles).
constexpr int kRepackSources = 256;
template <int CB = 0, int CR = 32>
__global__ __launch_bounds__(256) void k_repack(const float *__restrict__ sfm, float *__restrict__ dfm, int N,
                                                const int *__restrict__ src, const int *__restrict__ npos,
                                                const unsigned *__restrict__ seglive, const int *__restrict__ cols,
                                                int ncols, unsigned char *__restrict__ dcodes, unsigned *__restrict__ gd,
                                                int *__restrict__ overflow) {
  __shared__ int otile[32];            // distinct old tiles of this new tile
  __shared__ unsigned omask[32];       // their slots that this new tile takes
  __shared__ unsigned char bslot[32][32];  // old tile i, old slot s -> new slot
  __shared__ int nold;
  __shared__ unsigned segw[32];        // seglive words of the old tiles for the current 32 sources
  __shared__ float stage[32][33];
  static_assert(CB == 0 || CB == 1, "fp32 tiles or one-byte codes");
  constexpr int CE = CB > 0 ? kCacheEntries : 2;
  __shared__ __align__(8) unsigned dlk[CE];  // the dictionary's LDS cache (CB > 0)
  __shared__ __align__(8) unsigned dlc[CE];
  __shared__ int stop;
  if constexpr (CB > 0) {
    for (int i = threadIdx.x; i < CE; i += blockDim.x) dlk[i] = kDictEmpty;
  }
  const int R = *npos;
  // (codes: every 32-position tile of the last code tile, those past the list all zero)
  const int ntiles = CB > 0 ? (R + CR - 1) / CR * (CR / 32) : (R + 31) / 32;
  const int nkc = (ncols + kRepackSources - 1) / kRepackSources;
  const int tid = threadIdx.x, kk = tid >> 3, q = tid & 7;
  const int NW = (N + 31) / 32;
  for (int item = blockIdx.x; item < ntiles * nkc; item += gridDim.x) {
    const int t = item / nkc, k0 = (item % nkc) * kRepackSources;
    const int nb = max(0, min(32, R - t * 32));
    if constexpr (CB > 0) {
      if (tid == 0) stop = __hip_atomic_load(overflow, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __syncthreads();
      if (stop) return;  // uniform: every thread read the one word
    }
    if (tid == 0) {
      int n = 0, last = -1;
      for (int b = 0; b < nb; ++b) {
        const int sp = src[t * 32 + b];
        const int ot = sp >> 5;
        if (ot != last) {
          otile[n] = ot;
          omask[n] = 0u;
          ++n;
          last = ot;
        }
        omask[n - 1] |= 1u << (sp & 31);
        bslot[n - 1][sp & 31] = (unsigned char)b;
      }
      nold = n;
    }
    __syncthreads();
    const int n = nold;
    for (int kb = 0; kb < kRepackSources; kb += 32) {
      const int kp = k0 + kb + kk;  // source position; the source is cols[kp] with a column list
      const int k = kp < ncols ? (cols ? cols[kp] : kp) : N;
      // rows not taken from any old tile (past nb) stay zero
      for (int i = tid; i < 32 * 32; i += blockDim.x) stage[i >> 5][i & 31] = 0.0f;
      // k0 + kb is a multiple of 32: one bitmap word per old tile covers these sources, bit kk
      if (tid < n) segw[tid] = seglive ? seglive[(size_t)otile[tid] * NW + ((k0 + kb) >> 5)] : ~0u;
      __syncthreads();
      if (k < N) {
        // old tiles in batches of 8: the batch's loads are all issued before the first is used
        for (int i0 = 0; i0 < n; i0 += 8) {
          float4 v[8];
          unsigned mm[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int i = min(i0 + u, n - 1);
            mm[u] = i0 + u < n && ((segw[i] >> kk) & 1u) ? (omask[i] >> (4 * q)) & 15u : 0u;
            // without a branch: a quad that is not needed reads the first one of the old tiles
            // instead (a cache hit), so the eight loads issue back to back
            const size_t at = mm[u] ? ((size_t)otile[i] * N + k) * 32 : 0;
            v[u] = *(reinterpret_cast<const float4 *>(sfm + at) + q);
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            if (!mm[u]) continue;
            const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
            for (int c = 0; c < 4; ++c)
              if ((mm[u] >> c) & 1u) stage[kk][bslot[i0 + u][4 * q + c]] = e[c];
          }
        }
      }
      __syncthreads();
      if constexpr (CB > 0) {
        if (k < N) {
          // codes of rows 4q .. 4q + 3 of this 32-position tile, at its place in its code tile
          unsigned c[4];
          bool miss = false;
#pragma unroll
          for (int u = 0; u < 4; ++u) miss |= !cache_lookup(__float_as_uint(stage[kk][4 * q + u]), dlk, dlc, &c[u]);
          if (miss) {
#pragma unroll
            for (int u = 0; u < 4; ++u) c[u] = dict_code(stage[kk][4 * q + u], dlk, dlc, gd, overflow);
          }
          unsigned char *d = dcodes + ((size_t)(t / (CR / 32)) * N + k) * CR + (t % (CR / 32)) * 32 + 4 * q;
          *reinterpret_cast<unsigned *>(d) = c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24);
        }
      } else if (k < N) {
        *reinterpret_cast<float4 *>(dfm + ((size_t)t * N + k) * 32 + 4 * q) =
            make_float4(stage[kk][4 * q], stage[kk][4 * q + 1], stage[kk][4 * q + 2], stage[kk][4 * q + 3]);
      }
      __syncthreads();
    }
  }
}

// Layer-0 inputs as bits (the challenge inputs are binary images, Sec. IV): pack the live rows into
// feature-major bit tiles, bits[t][k] bit b = (Y[ids[t*T + b]][k] != 0). Any entry other than 0
// and 1 (or not finite) sets *nonbinary, and the bit route is then not used. Rows with a nonzero
// entry are recorded in rownz. One wave per (tile, run of kPackBlocks blocks of sources): with
// N % 4 == 0 a lane takes 4 consecutive sources per block (16-byte loads, 256 sources per block),
// otherwise one (64 per block). The rows' nonzero bits are gathered over the run and stored once.
constexpr int kPackBlocks = 16;
template <int T>
__global__ __launch_bounds__(256) void k_pack_bits(const float *__restrict__ yin, typename BitWord<T>::type *__restrict__ bits,
                                                   int N, const int *__restrict__ ids, const int *__restrict__ count,
                                                   int *__restrict__ rownz, int *__restrict__ nonbinary) {
  using W = typename BitWord<T>::type;
  const int R = *count;
  const int ntiles = (R + T - 1) / T;
  const bool vec = (N & 3) == 0;
  const int per_lane = vec ? 4 : 1;
  const int kblocks = (N + 64 * per_lane - 1) / (64 * per_lane);
  const int runs = (kblocks + kPackBlocks - 1) / kPackBlocks;
  const int lane = threadIdx.x & 63;
  const long long nwaves = (long long)gridDim.x * (blockDim.x >> 6);
  bool bad = false;
  for (long long item = blockIdx.x * (long long)(blockDim.x >> 6) + (threadIdx.x >> 6);
       item < (long long)ntiles * runs; item += nwaves) {
    const int t = (int)(item / runs), run = (int)(item % runs);
    const int nvalid = min(T, R - t * T);
    // row starts in units of 4 floats (vec) or floats: below 2^32 for any row id and width
    unsigned rowq[T];
#pragma unroll
    for (int b = 0; b < T; ++b) rowq[b] = (unsigned)ids[t * T + min(b, nvalid - 1)] * (unsigned)(vec ? N / 4 : N);
    const float4 *y4 = reinterpret_cast<const float4 *>(yin);
    unsigned rows_nz = 0u;
    const int kb_end = min(kblocks, (run + 1) * kPackBlocks);
    for (int kb = run * kPackBlocks; kb < kb_end; ++kb) {
      if (vec) {
        const int k = (kb * 64 + lane) * 4;
        const bool kin = k < N;
        unsigned word[4] = {0u, 0u, 0u, 0u};
        // rows in groups of 16 keep the loads in flight within the register budget
#pragma unroll
        for (int b0 = 0; b0 < T; b0 += 16) {
          float4 v[16];
#pragma unroll
          for (int b = 0; b < 16; ++b)
            v[b] = (b0 + b < nvalid && kin) ? load_stream_f4(y4 + rowq[b0 + b] + (k >> 2)) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int b = 0; b < 16; ++b) {
            const float e[4] = {v[b].x, v[b].y, v[b].z, v[b].w};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              const bool nz = e[c] != 0.0f;
              bad |= nz && e[c] != 1.0f;
              word[c] |= (unsigned)nz << (b0 + b);
            }
          }
        }
        rows_nz |= word[0] | word[1] | word[2] | word[3];
        if (kin) {
          W *dst = bits + (size_t)t * N + k;
          if constexpr (sizeof(W) == 2) {
            *reinterpret_cast<uint2 *>(dst) = make_uint2(word[0] | (word[1] << 16), word[2] | (word[3] << 16));
          } else {
            *reinterpret_cast<uint4 *>(dst) = make_uint4(word[0], word[1], word[2], word[3]);
          }
        }
      } else {
        const int k = kb * 64 + lane;
        const bool kin = k < N;
        float v[T];
#pragma unroll
        for (int b = 0; b < T; ++b) v[b] = (b < nvalid && kin) ? yin[(size_t)rowq[b] + k] : 0.0f;
        unsigned word = 0u;
#pragma unroll
        for (int b = 0; b < T; ++b) {
          const bool nz = v[b] != 0.0f;
          bad |= nz && v[b] != 1.0f;
          word |= (unsigned)nz << b;
        }
        rows_nz |= word;
        if (kin) bits[(size_t)t * N + k] = (W)word;
      }
    }
    // rows with a nonzero anywhere in this run: OR over the wave, then lane b stores row b's flag
    unsigned all = rows_nz;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) all |= __shfl_xor(all, d, 64);
    if (lane < nvalid && ((all >> lane) & 1u)) rownz[ids[t * T + lane]] = 1;
  }
  if (__ballot(bad) && lane == 0) *nonbinary = 1;
}

// (byte k of u) & 0xF0 in one instruction: a bitwise and whose first operand is byte k of u (a
// byte-select on the operand); f0 holds 0xF0.
__device__ __forceinline__ unsigned byte_and_f0(unsigned u, int k, unsigned f0) {
  unsigned r;
  switch (k) {
    case 0: return u & 0xF0u;
    case 1:
      asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD"
          : "=v"(r) : "v"(u), "v"(f0));
      return r;
    case 2:
      asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD"
          : "=v"(r) : "v"(u), "v"(f0));
      return r;
    default:
      asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD"
          : "=v"(r) : "v"(u), "v"(f0));
      return r;
  }
}

// Layer 0 from bit tiles of T rows (T = 16 or 32): every term is fma(bit, w, acc) with bit 0 or 1,
// the same fp32 chain as the general kernels since 1*w and 0*w are exact. blockDim kBitsThreads. LDS
// holds the tile's N words and a table that turns 4 input bits into as many floats (16
// entries of 4 floats: few distinct entries, so a wave's reads of it are mostly broadcasts). Lane =
// output j; each lane carries the T rows of its output, so one ELL entry and one word serve T
// edge-rows; for 16-row tiles the table reads of a term are issued one term ahead. Results
// go to feature-major tiles of 32 rows (list position p at tile p / 32, slot p % 32): a lane writes
// its T rows of output j as T / 4 16-byte stores. Slots past the list's end get zeros.
// ell is the layer's ELL with source k given as k * sizeof(word), the byte offset of its word in
// the bit tile (LayerDev::ellw).
// KC = 32: the 32 ELL entries of a lane's output are all loaded before the first term is used.
// CODES: instead of fp32 values, write each output's one-byte code in the value dictionary gd
// (same tile layout, one byte per row); a full dictionary sets *overflow. With *skip set (an input
// that is not 0 or 1) the kernel does nothing.
template <int T, int KC, bool CODES>
__global__ __launch_bounds__(kBitsThreads) void k_layer_bits(const typename BitWord<T>::type *__restrict__ bits,
                                                     float *__restrict__ fout, int N, const int2 *__restrict__ ell,
                                                     int K, const float *__restrict__ bias,
                                                     float ymax, const int *__restrict__ count,
                                                     unsigned *__restrict__ masks, unsigned *__restrict__ gd,
                                                     int *__restrict__ overflow, const int *__restrict__ skip) {
  if (*skip) return;  // an input is not 0 or 1 (found by k_pack_bits): the layer goes another way
  constexpr int CR = code_rows(T);
  using W = typename BitWord<T>::type;
  const unsigned f0 = 0xF0u;                            // the byte-select ands' mask, in a register
  // static LDS (addresses known at compile time, so they fold into the instructions' offsets): the
  // table, the tile's live-row mask and the dictionary cache; dynamic LDS: the tile
  // one struct fixes the layout: the table at LDS address 0 and the tile after the small arrays,
  // so that every LDS address here is a register plus a constant that fits the instruction offset
  struct BitsLds {
    float4 lut[kLutF4];
    unsigned dlk[kCacheEntries];
    unsigned dlc[kCacheEntries];
    unsigned tilemask;
    unsigned pad[3];
    W tile[bits_tile_bytes(T) / sizeof(W)];
  };
  __shared__ __align__(16) BitsLds sm;
  float4 *const lut = sm.lut;
  unsigned *const dlk = sm.dlk;
  unsigned *const dlc = sm.dlc;
  unsigned &tilemask = sm.tilemask;
  W *const tile = sm.tile;
  const int R = *count;
  const int ntiles = (R + T - 1) / T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int blocks = (N + 63) / 64;                 // output blocks of 64
  const int rounds = (blocks + nw - 1) / nw;        // rounds of one block per wave
  // Every tile's outputs in 8 chunks, item w taking chunk w % 8: with the grid a multiple of 8, that
  // is the XCD the workgroup runs on, so each XCD reads one eighth of the layer's ELL (2.1 MB at
  // 65536 neurons), which stays in its L2 while every tile passes; with whole tiles per workgroup
  // each tile re-read the whole ELL (16.8 MB) through the L2s, tens of GB per layer. A tile is then
  // staged 8 times (its bits are 1/16 of the ELL's bytes at 16 rows).
  const Chunking ch = chunking(ntiles, rounds, gridDim.x % 8 == 0 ? 8 : 1);
  // codes with whole tiles as items: keep the tiles of one code group on one XCD
  const bool grouped = CODES && ch.nchunks == 1 && gridDim.x % (8 * (CR / T)) == 0;
  const int items = grouped ? (ntiles + gridDim.x - 1) / gridDim.x * gridDim.x : ntiles * ch.nchunks;
  for (int i = tid; i < kLutF4; i += blockDim.x)
    lut[i] = make_float4((float)(i & 1), (float)((i >> 1) & 1), (float)((i >> 2) & 1), (float)((i >> 3) & 1));
  if (tid == 0) tilemask = 0u;
  if (CODES)
    for (int i = tid; i < kCacheEntries; i += blockDim.x) dlk[i] = kDictEmpty;
  for (int w = blockIdx.x; w < items; w += gridDim.x) {
    const int t = grouped ? code_group_tile(w, CR / T) : w / ch.nchunks;
    const int c = grouped ? 0 : w % ch.nchunks;
    if (t >= ntiles) continue;  // uniform over the workgroup
    const int p0 = t * T;
    const int nvalid = min(T, R - p0);
    {
      const W *src = bits + (size_t)t * N;
      if ((reinterpret_cast<uintptr_t>(src) & 15) == 0) {
        const int n16 = (int)(((size_t)N * sizeof(W)) / 16);
        for (int i = tid; i < n16; i += blockDim.x) reinterpret_cast<int4 *>(tile)[i] = reinterpret_cast<const int4 *>(src)[i];
        for (int k = n16 * (int)(16 / sizeof(W)) + tid; k < N; k += blockDim.x) tile[k] = src[k];
      } else {
        for (int k = tid; k < N; k += blockDim.x) tile[k] = src[k];
      }
    }
    __syncthreads();
    const char *tb = reinterpret_cast<const char *>(tile);
    unsigned live = 0u;
    const int r_end = min(rounds, (c + 1) * ch.rounds_per_chunk);
    const unsigned ell_row = (unsigned)N * (unsigned)sizeof(int2);  // bytes per ELL slot
    const __amdgpu_buffer_rsrc_t ersrc = buffer_rsrc(ell, (unsigned)K * ell_row);
    for (int r = c * ch.rounds_per_chunk; r < r_end; ++r) {
      const int blk = r * nw + wave;
      if (blk >= blocks) break;
      const int j = blk * 64 + lane;
      const bool jin = j < N;
      // ELL entries by buffer loads: the lane's offset in a vector register, the slot's offset
      // (sl * N * 8) in a scalar one, so that no vector instruction forms an address
      const unsigned jo8 = (jin ? (unsigned)j : 0u) * (unsigned)sizeof(int2);
      auto ej = [&](int sl) {
        return __builtin_bit_cast(int2, __builtin_amdgcn_raw_buffer_load_b64(ersrc, jo8, (unsigned)sl * ell_row, 0));
      };
      float acc[T];
#pragma unroll
      for (int b = 0; b < T; ++b) acc[b] = 0.0f;
      // the source's word gives the T input bits; each nibble picks four floats (0 or 1) from the
      // table
      auto expand = [&](unsigned word, float4 (&v)[T / 4]) {
        // byte offset of nibble 2k's entry: byte k of (word << 4) with its low 4 bits cleared; of
        // nibble 2k + 1's: byte k of word, likewise (one byte-select and per nibble)
        const unsigned x = word << 4;
        const char *lb = reinterpret_cast<const char *>(lut);
#pragma unroll
        for (int k = 0; k < T / 8; ++k) {
          v[2 * k] = *reinterpret_cast<const float4 *>(lb + byte_and_f0(x, k, f0));
          v[2 * k + 1] = *reinterpret_cast<const float4 *>(lb + byte_and_f0(word, k, f0));
        }
      };
      auto apply = [&](const float4 (&v)[T / 4], float wv) {
#pragma unroll
        for (int n = 0; n < T / 4; ++n) {
          acc[4 * n] = fmaf(v[n].x, wv, acc[4 * n]);
          acc[4 * n + 1] = fmaf(v[n].y, wv, acc[4 * n + 1]);
          acc[4 * n + 2] = fmaf(v[n].z, wv, acc[4 * n + 2]);
          acc[4 * n + 3] = fmaf(v[n].w, wv, acc[4 * n + 3]);
        }
      };
      if constexpr (KC > 0) {
        // slots go in groups of 16 with the issue order pinned by scheduling barriers: a group's
        // tile words are read while the next group's ELL entries load, then its terms run
        // slots in groups of G (16 rows: 16 with the table reads one term ahead; 32 rows: 8, reads
        // not ahead, which keeps the lane within 128 registers)
        constexpr int G = T == 16 ? 16 : 8;
        constexpr bool AHEAD = T == 16;
        static_assert(KC % G == 0, "KC must be a multiple of the group");
        int2 e[G];
#pragma unroll
        for (int i = 0; i < G; ++i) e[i] = ej(i);
#pragma unroll
        for (int h = 0; h < KC; h += G) {
          mem_fence_compiler();
          unsigned wd[G];
          float wv[G];
#pragma unroll
          for (int i = 0; i < G; ++i) {
            wd[i] = *reinterpret_cast<const W *>(tb + (unsigned)e[i].x);
            wv[i] = __int_as_float(e[i].y);
          }
          if (h + G < KC) {
#pragma unroll
            for (int i = 0; i < G; ++i) e[i] = ej(h + G + i);
          }
          mem_fence_compiler();
          if constexpr (AHEAD) {
            // table reads run one term ahead of the fmas (two buffers by parity: no copies)
            float4 vb[2][T / 4];
            expand(wd[0], vb[0]);
#pragma unroll
            for (int i = 0; i < G; ++i) {
              if (i + 1 < G) expand(wd[i + 1], vb[(i + 1) & 1]);
              apply(vb[i & 1], wv[i]);
              // this term's fmas complete here, and the next table reads are issued after them
#pragma unroll
              for (int b = 0; b < T; b += 4) pin4(acc[b], acc[b + 1], acc[b + 2], acc[b + 3]);
              mem_fence_compiler();
            }
          } else {
#pragma unroll
            for (int i = 0; i < G; ++i) {
              float4 v[T / 4];
              expand(wd[i], v);
              apply(v, wv[i]);
#pragma unroll
              for (int b = 0; b < T; b += 4) pin4(acc[b], acc[b + 1], acc[b + 2], acc[b + 3]);
              mem_fence_compiler();
            }
          }
        }
      } else {
        for (int sl = 0; sl < K; ++sl) {
          const int2 e = ej(sl);
          float4 v[T / 4];
          expand(*reinterpret_cast<const W *>(tb + (unsigned)e.x), v);
          apply(v, __int_as_float(e.y));
        }
      }
      if (jin) {
        // rows past nvalid have all-zero bits, so their outputs are zeros
        const float bj = bias[j];
        if constexpr (CODES) {
          uint4 *dst = reinterpret_cast<uint4 *>(reinterpret_cast<unsigned char *>(fout) +
                                                 ((size_t)(p0 / CR) * N + j) * CR + p0 % CR);
          // every row's value (in place of its accumulator), then per 16 rows the LDS cache's codes;
          // the full lookup (global table included) only on a lane where one of them missed
#pragma unroll
          for (int u = 0; u < T; ++u) {
            acc[u] = activate(acc[u], bj, ymax);
            live |= (acc[u] > 0.0f ? 1u : 0u) << u;
          }
          unsigned cw[T / 4];
          // rows [R0, R0 + 16), R0 a compile-time constant (so that every array index is one)
          auto encode16 = [&](auto r0c) {
            constexpr int R0 = decltype(r0c)::value;
            unsigned code[16];
            bool miss = false;
#pragma unroll
            for (int u = 0; u < 16; ++u) miss |= !cache_lookup(__float_as_uint(acc[R0 + u]), dlk, dlc, &code[u]);
            if (miss) {
#pragma unroll
              for (int u = 0; u < 16; ++u) code[u] = dict_code(acc[R0 + u], dlk, dlc, gd, overflow);
            }
#pragma unroll
            for (int n = 0; n < 4; ++n)
              cw[R0 / 4 + n] = code[4 * n] | (code[4 * n + 1] << 8) | (code[4 * n + 2] << 16) | (code[4 * n + 3] << 24);
          };
          encode16(std::integral_constant<int, 0>{});
          if constexpr (T == 32) encode16(std::integral_constant<int, 16>{});
#pragma unroll
          for (int n = 0; n < T / 16; ++n) dst[n] = make_uint4(cw[4 * n], cw[4 * n + 1], cw[4 * n + 2], cw[4 * n + 3]);
          // the rest of the last code tile gets code 0 (+0.0)
          if (t + 1 == ntiles)
            for (int n = T / 16; n < (CR - p0 % CR) / 16; ++n) dst[n] = make_uint4(0u, 0u, 0u, 0u);
        } else {
          float4 *dst = reinterpret_cast<float4 *>(fout + ((size_t)(p0 >> 5) * N + j) * 32 + (p0 & 31));
#pragma unroll
          for (int n = 0; n < T / 4; ++n) {
            const float4 y = make_float4(activate(acc[4 * n], bj, ymax), activate(acc[4 * n + 1], bj, ymax),
                                         activate(acc[4 * n + 2], bj, ymax), activate(acc[4 * n + 3], bj, ymax));
            dst[n] = y;
            live |= ((y.x > 0.0f ? 1u : 0u) | (y.y > 0.0f ? 2u : 0u) | (y.z > 0.0f ? 4u : 0u) | (y.w > 0.0f ? 8u : 0u))
                    << (4 * n);
          }
          if (T == 16 && (p0 & 31) == 0 && t + 1 == ntiles) {
            // the last 32-row tile has no second half: zero its slots 16..31
#pragma unroll
            for (int n = 0; n < 4; ++n) dst[4 + n] = make_float4(0.f, 0.f, 0.f, 0.f);
          }
        }
      }
    }
    if (live) atomicOr(&tilemask, live);
    __syncthreads();
    if (tid == 0) {
      unsigned m = tilemask;
      tilemask = 0u;
      m &= nvalid >= 32 ? 0xffffffffu : ((1u << nvalid) - 1u);
      if (m) atomicOr(&masks[p0 >> 5], m << (p0 & 31));
    }
    __syncthreads();
  }
}

// Dictionary of a uniform layer on binary inputs (every column K sources, weight w, bias b): a
// column with c sources at 1 has z = z_c, the fp32 chain of c fma(1, w, .) steps from +0 (the steps
// with input 0 leave the accumulator unchanged: fma(0, w, acc) = acc since acc is never -0), so its
// output is dict[c] = activate(z_c, b). Codes c in [0, K]; the other slots are left free.
// misc[kCountMinSlot] receives the smallest c with dict[c] > 0 (K + 1 if none; with w > 0 the
// outputs grow with c, so a row is live exactly when one of its counts reaches it).
constexpr int kCountMinSlot = 3;
__global__ void k_count_dict(unsigned *__restrict__ dict, int *__restrict__ misc, int K, float w, float b,
                             float ymax) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  float z = 0.0f;
  int cmin = K + 1;
  for (int c = 0; c <= K; ++c) {
    const float y = activate(z, b, ymax);
    dict[c] = __float_as_uint(y);
    if (y > 0.0f && cmin > K) cmin = c;
    z = fmaf(1.0f, w, z);
  }
  misc[kCountMinSlot] = cmin;
}

// Carry-save adder on bit-sliced words: per bit position, a + b + c = sum + 2 * carry.
__device__ __forceinline__ void csa(unsigned &carry, unsigned &sum, unsigned a, unsigned b, unsigned c) {
  carry = __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);  // majority
  sum = __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);    // three-way xor
}

// Layer 0 of a uniform layer (K = 32, w > 0) on bit tiles of T rows: for each output, the counts
// of set input bits among its 32 sources, for all rows of a word at once. The 32 source words go
// through a carry-save adder tree (two 16-word blocks), giving the six bit planes of the counts
// (0..32); a bit-sliced comparison with the first live count gives the live rows, and a transpose
// turns the planes into one byte per row: the output's code, decoded by the dictionary of
// k_count_dict. blockDim 1024; lane = output (T = 32) or outputs j and j + 64 in the low and high
// halves of each word (T = 16). LDS holds the tile's N words; the source indices are read 8 per
// 16-byte load from the [4][N][8] u16 table. Codes go to tiles of CR rows, one byte per row. With
// ROWMAJOR (T = 32; widths staged in LDS) the outputs are decoded instead and written as fp32 rows,
// yout[ids[p]][j] = dict[code] (the dictionary is copied after the tile in LDS). With cols set, only
// the ncols columns cols[p] are computed, their source lists in ell16 as [4][ncols][8].
template <int T, bool ROWMAJOR>
__global__ __launch_bounds__(1024) void k_layer_count(const typename BitWord<T>::type *__restrict__ bits,
                                                      unsigned char *__restrict__ cout, int N,
                                                      const uint4 *__restrict__ ell16, const int *__restrict__ misc,
                                                      const int *__restrict__ count, unsigned *__restrict__ masks,
                                                      float *__restrict__ yout, const int *__restrict__ ids,
                                                      const unsigned *__restrict__ dict, const int *__restrict__ cols,
                                                      int ncols, const int *__restrict__ skip) {
  static_assert(!ROWMAJOR || T == 32, "rows of fp32 outputs from 32-row bit tiles");
  if (*skip) return;  // an input is not 0 or 1 (found by k_pack_bits): the layer goes another way
  constexpr int CR = code_rows(T);
  using W = typename BitWord<T>::type;
  constexpr int OPL = T == 16 ? 2 : 1;  // outputs per lane
  extern __shared__ float4 smem[];
  unsigned &tilemask = *reinterpret_cast<unsigned *>(smem);
  W *tile = reinterpret_cast<W *>(smem + 1);
  // ROWMAJOR: the dictionary, then the tile's row ids, after the tile's words
  float *dl = reinterpret_cast<float *>(tile + ((N + 3) / 4) * 4);
  int *rid = reinterpret_cast<int *>(dl + kDictSlots);
  if constexpr (ROWMAJOR)
    for (int i = threadIdx.x; i < kDictSlots; i += blockDim.x) dl[i] = __uint_as_float(dict[i]);
  const int R = *count;
  const int cmin = misc[kCountMinSlot];
  const int ntiles = (R + T - 1) / T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int blocks = (ncols + 64 * OPL - 1) / (64 * OPL);  // output blocks of one wave
  const int rounds = (blocks + nw - 1) / nw;
  const Chunking ch = chunking(ntiles, rounds);
  // whole tiles as items: keep the tiles of one code group on one XCD
  const bool grouped = ch.nchunks == 1 && gridDim.x % (8 * (CR / T)) == 0;
  const int items = grouped ? (ntiles + gridDim.x - 1) / gridDim.x * gridDim.x : ntiles * ch.nchunks;
  if (tid == 0) tilemask = 0u;
  for (int w = blockIdx.x; w < items; w += gridDim.x) {
    const int t = grouped ? code_group_tile(w, CR / T) : w / ch.nchunks;
    const int c = grouped ? 0 : w % ch.nchunks;
    if (t >= ntiles) continue;  // uniform over the workgroup
    const int p0 = t * T;
    const int nvalid = min(T, R - p0);
    {
      const W *src = bits + (size_t)t * N;
      if ((reinterpret_cast<uintptr_t>(src) & 15) == 0) {
        const int n16 = (int)(((size_t)N * sizeof(W)) / 16);
        for (int i = tid; i < n16; i += blockDim.x) reinterpret_cast<int4 *>(tile)[i] = reinterpret_cast<const int4 *>(src)[i];
        for (int k = n16 * (int)(16 / sizeof(W)) + tid; k < N; k += blockDim.x) tile[k] = src[k];
      } else {
        for (int k = tid; k < N; k += blockDim.x) tile[k] = src[k];
      }
    }
    if constexpr (ROWMAJOR)
      if (threadIdx.x < T) rid[threadIdx.x] = (int)threadIdx.x < nvalid ? ids[p0 + threadIdx.x] : -1;
    __syncthreads();
    unsigned live = 0u;
    const int r_end = min(rounds, (c + 1) * ch.rounds_per_chunk);
    for (int r = c * ch.rounds_per_chunk; r < r_end; ++r) {
      const int blk = r * nw + wave;
      if (blk >= blocks) break;
      int jo[OPL], jc[OPL];  // output position and its column
      bool jin[OPL];
#pragma unroll
      for (int u = 0; u < OPL; ++u) {
        jo[u] = blk * 64 * OPL + u * 64 + lane;
        jin[u] = jo[u] < ncols;
        jc[u] = cols ? cols[min(jo[u], ncols - 1)] : jo[u];
      }
      // the 32 source indices of each output, 8 per load (positions past the last read the last)
      uint4 ix[OPL][4];
#pragma unroll
      for (int u = 0; u < OPL; ++u)
#pragma unroll
        for (int g = 0; g < 4; ++g) ix[u][g] = ell16[(size_t)g * ncols + min(jo[u], ncols - 1)];
      auto word = [&](int sl) -> unsigned {
        unsigned x = 0u;
#pragma unroll
        for (int u = 0; u < OPL; ++u) {
          const uint4 q = ix[u][sl >> 3];
          const unsigned pr = ((sl & 7) < 4) ? ((sl & 7) < 2 ? q.x : q.y) : ((sl & 7) < 6 ? q.z : q.w);
          const unsigned k = (sl & 1) ? (pr >> 16) : (pr & 0xffffu);
          x |= (unsigned)tile[k] << (16 * u);
        }
        return x;
      };
      // carry-save adder tree over two blocks of 16 source words
      unsigned ones = 0u, twos = 0u, fours = 0u, eights = 0u, s16[2];
#pragma unroll
      for (int blk16 = 0; blk16 < 2; ++blk16) {
        const int b0 = 16 * blk16;
        unsigned twosA, twosB, foursA, foursB, eightsA, eightsB;
        csa(twosA, ones, ones, word(b0 + 0), word(b0 + 1));
        csa(twosB, ones, ones, word(b0 + 2), word(b0 + 3));
        csa(foursA, twos, twos, twosA, twosB);
        csa(twosA, ones, ones, word(b0 + 4), word(b0 + 5));
        csa(twosB, ones, ones, word(b0 + 6), word(b0 + 7));
        csa(foursB, twos, twos, twosA, twosB);
        csa(eightsA, fours, fours, foursA, foursB);
        csa(twosA, ones, ones, word(b0 + 8), word(b0 + 9));
        csa(twosB, ones, ones, word(b0 + 10), word(b0 + 11));
        csa(foursA, twos, twos, twosA, twosB);
        csa(twosA, ones, ones, word(b0 + 12), word(b0 + 13));
        csa(twosB, ones, ones, word(b0 + 14), word(b0 + 15));
        csa(foursB, twos, twos, twosA, twosB);
        csa(eightsB, fours, fours, foursA, foursB);
        csa(s16[blk16], eights, eights, eightsA, eightsB);
      }
      const unsigned pl[6] = {ones, twos, fours, eights, s16[0] ^ s16[1], s16[0] & s16[1]};
      // rows whose count reaches cmin (bit-sliced comparison from the top plane down)
      unsigned gt = 0u, eq = 0xffffffffu;
#pragma unroll
      for (int i = 5; i >= 0; --i) {
        if ((cmin >> i) & 1) {
          eq &= pl[i];
        } else {
          gt |= eq & pl[i];
          eq &= ~pl[i];
        }
      }
      const unsigned ge = cmin > 63 ? 0u : (gt | eq);
      // transpose the planes into one byte per row: dword d holds rows 4d..4d+3
      unsigned cw[8];
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        unsigned acc = 0u;
#pragma unroll
        for (int i = 0; i < 6; ++i) {
          const unsigned nib = (pl[i] >> (4 * d)) & 15u;
          acc |= ((nib * 0x00204081u) & 0x01010101u) << i;
        }
        cw[d] = acc;
      }
#pragma unroll
      for (int u = 0; u < OPL; ++u) {
        if (!jin[u]) continue;
        const unsigned rows = T == 16 ? ((ge >> (16 * u)) & 0xffffu) : ge;
        live |= rows;
        if constexpr (ROWMAJOR) {
          // row b's code is byte b % 4 of cw[b / 4]; rows past the list are not written
#pragma unroll
          for (int b = 0; b < T; ++b) {
            const int row = rid[b];
            if (row >= 0) yout[(size_t)row * N + jc[u]] = dl[(cw[b >> 2] >> (8 * (b & 3))) & 255u];
          }
          continue;
        }
        uint4 *dst = reinterpret_cast<uint4 *>(cout + ((size_t)(p0 / CR) * N + jc[u]) * CR + p0 % CR);
        // plain stores: the tiles of one code group fill each segment in parts, merged in L2
        if (T == 32) {
          dst[0] = make_uint4(cw[0], cw[1], cw[2], cw[3]);
          dst[1] = make_uint4(cw[4], cw[5], cw[6], cw[7]);
        } else {
          dst[0] = make_uint4(cw[4 * u], cw[4 * u + 1], cw[4 * u + 2], cw[4 * u + 3]);
        }
        // the rest of the last code tile gets code 0 (+0.0)
        if (t + 1 == ntiles)
          for (int n = T / 16; n < (CR - p0 % CR) / 16; ++n) dst[n] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
    if (live) atomicOr(&tilemask, live);
    __syncthreads();
    if (tid == 0) {
      unsigned m = tilemask;
      tilemask = 0u;
      m &= nvalid >= 32 ? 0xffffffffu : ((1u << nvalid) - 1u);
      if (m) atomicOr(&masks[p0 >> 5], m << (p0 & 31));
    }
    __syncthreads();
  }
}

// The workspace of sdnn_infer_static: a file-scope array in device memory, 64 MiB, of which each
// device that loads the library holds its own copy until the process ends. Host code never passes
// the array's name to a kernel or a copy (on the host it is a stand-in, not a device address): it
// uses the address hipGetSymbolAddress returns for the current device, looked up once per device.
constexpr size_t kStaticWorkspaceBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device`, which must be the current device.
sdnn_status scratch_address(int device, void **out) {
  if (device < 0 || device >= kMaxDevices) return fail(SDNN_EINVAL, "device %d out of range", device);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(SDNN_EDEVICE, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    }
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return SDNN_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------------
// Host side

struct LayerDev {
  const int2 *ell = nullptr;
  // layer 0 of the global-tile path (bit route): the ELL with each source given as the byte offset
  // of its word in a bit tile (source k * sizeof(word)) instead of its offset in a 32-row fp32 tile
  const int2 *ellw = nullptr;
  const float *bias = nullptr;
  int K = 0;
  // uniform layer (set only with the opt-in equal-value kernels): every column holds exactly K
  // sources, all weights are w and all biases b
  bool uniform = false;
  float w = 0.0f, b = 0.0f;
  // layer with K == 32 on widths staged in LDS, and uniform layer 0 of any width: [K/8][N][8] u16
  // source indices, eight per 16-byte load; unless the layer is uniform, its weights in the same
  // grouping, [K/8][N][8] fp32 (w8)
  const uint4 *ell16 = nullptr;
  const float *w8 = nullptr;
  // LDS row placement for k_layer_lds (path 0, the first kPlacedLayers layers with ell16): neuron k
  // of the layer's input is staged at tile row place[k], and pell16 is ell16 with every source k
  // replaced by place[k] (see bank_placement)
  const unsigned short *place = nullptr;
  const uint4 *pell16 = nullptr;
  // global-tile path, layer with K == 32 and N <= 65536: [K][N] u16 source indices (the ELL's
  // sources), and unless the layer is uniform its weights [K][N] fp32 beside them (w32)
  const unsigned short *src16 = nullptr;
  const float *w32 = nullptr;
  // distinct columns (uniform layer with K == 32): columns with equal source lists have equal
  // outputs, so only the D representatives cols[0..D) need computing, with their source lists in
  // src16c ([K][D] u16, beside src16) and ell16c ([K/8][D][8], beside ell16). Usable (dedup_ok) once
  // the next layer's sources point to representatives only (or for the last layer).
  const int *cols = nullptr;
  const unsigned short *src16c = nullptr;
  const uint4 *ell16c = nullptr;
  // layer 0 of a uniform layer with K == 32: the lists of ell16 (and ell16c) with each column's
  // sources reordered for the counting kernel, whose counts do not depend on the order
  const uint4 *ell16s = nullptr, *ell16cs = nullptr;
  // widths staged in LDS: the positions of ell16 (and of ell16c) reordered for the fused kernel
  // with tiles of 4 << c rows (c = 0 also serves 1 and 2; see conflict_grouped_order): gcols[c][p]
  // is the column at position p, gell16[c] its sources
  const int *gcols[3] = {}, *gcolsc[3] = {};
  const uint4 *gell16[3] = {}, *gell16c[3] = {};
  const float *gw8[3] = {};  // the weights of gell16's positions (layers with w8)
  int D = 0;
  bool dedup_ok = false;
};

// Layers (from layer 0) that get an LDS row placement: the per-layer kernel runs the first layers
// of a batch, before the fused launch takes over.
constexpr int kPlacedLayers = 64;

// LDS row placement for k_layer_lds. The kernel reads a source's B rows (B * 4 bytes) with 16-byte
// lane reads; an LDS cycle serves 16 lanes (256 bytes, 64 banks), which are the G = 64 / B
// consecutive output columns of a group at one slot. Row r of the tile starts at bank (r B) mod 64,
// so the group's reads of distinct sources collide when their rows agree mod G; the cycles a read
// takes are the largest number of distinct sources on one residue. The sources of a column are
// fixed (and their order, which is the summation order), but the row of each neuron in the tile is
// free: this local search swaps the rows of two neurons whenever the summed cycles of the (group,
// slot) reads that involve them do not grow. h16: the layer's [4][N][8] source groups (ell16).
std::vector<uint16_t> bank_placement(const uint16_t *h16, int N, int B, uint64_t seed, int iters) {
  const int G = std::max(1, 64 / B);
  std::vector<uint16_t> place((size_t)N);
  for (int k = 0; k < N; ++k) place[(size_t)k] = (uint16_t)k;
  if (G < 2 || N < 2 * G) return place;
  auto srcof = [&](int j, int sl) { return (int)h16[((size_t)(sl / 8) * N + j) * 8 + sl % 8]; };
  const int ngroups = (N + G - 1) / G;
  // (group, slot) reads of each neuron, as a CSR over neurons
  std::vector<int> deg((size_t)N + 1, 0);
  for (int j = 0; j < N; ++j)
    for (int sl = 0; sl < 32; ++sl) ++deg[(size_t)srcof(j, sl) + 1];
  for (int k = 0; k < N; ++k) deg[(size_t)k + 1] += deg[(size_t)k];
  std::vector<int> occ((size_t)deg[(size_t)N]), fill(deg.begin(), deg.end() - 1);
  for (int j = 0; j < N; ++j)
    for (int sl = 0; sl < 32; ++sl) occ[(size_t)fill[(size_t)srcof(j, sl)]++] = (j / G) * 32 + sl;
  auto cycles = [&](int gs) {
    const int g = gs / 32, sl = gs % 32;
    int rows[64], n = 0, load[64] = {0}, m = 0;
    for (int j = g * G; j < std::min(N, g * G + G); ++j) {
      const int k = srcof(j, sl);
      bool dup = false;
      for (int t = 0; t < n; ++t) dup |= rows[t] == k;
      if (dup) continue;
      rows[n++] = k;
      m = std::max(m, ++load[place[(size_t)k] % G]);
    }
    return m;
  };
  (void)ngroups;
  uint64_t x = seed;
  auto next = [&]() {  // SplitMix64
    x += 0x9E3779B97F4A7C15ull;
    uint64_t z = x;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  };
  std::vector<int> touched;
  for (int it = 0; it < iters; ++it) {
    const int a = (int)(next() % (uint64_t)N), c = (int)(next() % (uint64_t)N);
    if (place[(size_t)a] % G == place[(size_t)c] % G) continue;
    touched.clear();
    for (int t = deg[(size_t)a]; t < deg[(size_t)a + 1]; ++t) touched.push_back(occ[(size_t)t]);
    for (int t = deg[(size_t)c]; t < deg[(size_t)c + 1]; ++t) touched.push_back(occ[(size_t)t]);
    std::sort(touched.begin(), touched.end());
    touched.erase(std::unique(touched.begin(), touched.end()), touched.end());
    int before = 0, after = 0;
    for (int gs : touched) before += cycles(gs);
    std::swap(place[(size_t)a], place[(size_t)c]);
    for (int gs : touched) after += cycles(gs);
    if (after > before) std::swap(place[(size_t)a], place[(size_t)c]);
  }
  return place;
}

}  // namespace

struct sdnn_net {
  int32_t N = 0, L = 0;
  float ymax = 32.0f;
  int path = 0;  // 0: LDS tiles, 1: global feature-major tiles
  int B = 0;     // rows per tile: LDS tile (path 0) or global feature-major tile (path 1)
  int bitsT = 0; // rows per layer-0 bit tile (path 1), 0 if the bit route is not available
  int device = -1;
  int cus = 0;
  bool poisoned = false;
  // kernels that exploit layers whose weights and biases are all equal (opt-in, before any load;
  // see sdnn_enable_equal_value_kernels)
  bool equal_value_kernels = false;
  std::vector<LayerDev> layers;
  std::vector<void *> allocations;
  // duplicate columns: representatives of the last layer loaded (rep[j] = smallest column with j's
  // source list), which the next layer's sources are mapped through when it is loaded right after
  std::vector<int32_t> prev_rep;
  int32_t prev_rep_layer = -1;
  std::vector<int32_t> last_rep;  // the same for layer L - 1 (final rows are expanded through it)
  // device tables of the layers, for launches that run several layers: one per fused tile height
  // class (4 << c rows; class 0 also for 1 and 2 rows)
  LayerPtr *lp_dev[3] = {};
  int32_t n_loaded = 0;
  // last run
  bool ran = false;
  int64_t M = 0;
  hipStream_t stream = nullptr;
  char *ws = nullptr;
  float *ybuf[2] = {nullptr, nullptr};  // path 0: row-major activations
  float *fm[2] = {nullptr, nullptr};    // path 1: feature-major tiles of 32 list positions
  int *ids[2] = {nullptr, nullptr};     // live lists: row id per position
  int *src[2] = {nullptr, nullptr};     // path 1: position in the previous list, per position
  unsigned *masks = nullptr;               // per-tile liveness bits (path 1: layers l % 3 == 0)
  unsigned *masks_rot[3] = {nullptr, nullptr, nullptr};  // path 1: layer l uses masks_rot[l % 3]
  int *rownz = nullptr, *counts = nullptr;
  int *misc = nullptr;  // device flags and counters: [0] a layer-0 input is not 0 or 1, [2] dictionary full,
                        // [4 + i] positions in list i
  unsigned *dict = nullptr;  // value dictionary of one-byte activation codes (kDictWords words; decoding reads the first 256)
  unsigned *dict16 = nullptr;  // path 1: the dictionary of two-byte codes (dict_words<2>() words)
  unsigned *seglive = nullptr;  // path 1: per fp32 tile, one bit per source: the segment was stored
  unsigned *part[2] = {nullptr, nullptr};  // path 1: partial liveness words of few-tile layers, by layer parity
  unsigned *spread = nullptr;              // path 1: liveness words of large layers, one 128-byte line each
  long long *final_ids = nullptr;
  int final_list = 0;        // which ids buffer holds the final list
  int32_t layers_run = 0;    // layers enqueued by the last infer
  std::vector<int32_t> layer_kernel, layer_launches;  // per layer of the last infer (sdnn_layer_info)
  const float *final_y = nullptr;   // path 0: final activations, row-major by row id
  const float *final_fm = nullptr;  // path 1: final activation tiles; live row i is at position src[final_list][i]
  int32_t *pinned = nullptr; // read-back slots (0-3: polling ring, 6: input-not-binary flag, 7: exact count)
  // progress word of few-tile layers, in coherent host memory written by the device (see
  // progress_word); progress_dev is its device address
  unsigned long long *progress = nullptr, *progress_dev = nullptr;
  // word in coherent host memory where a compaction reports its count and flags (see k_compact);
  // notify_dev is its device address, notify_seq the tag of the last report asked for
  unsigned long long *notify = nullptr, *notify_dev = nullptr;
  uint32_t notify_seq = 0;
  uint32_t run_gen = 0;      // generation of the current infer, in the progress word's top bits
  std::vector<hipEvent_t> events;
  // profiling
  bool profiling = false;
  int prof_mode = 0;              // 1: every layer, 2: large layers only
  std::vector<char> prof_rec;     // layers recorded by the last infer
  bool pending_times = false;
  std::vector<hipEvent_t> prof_start, prof_end;
  std::vector<double> prof_ms;
  std::vector<int64_t> prof_runs;
};

namespace {

#define HIP_OR_POISON(net, call)                                                                   \
  do {                                                                                             \
    hipError_t e_ = (call);                                                                        \
    if (e_ != hipSuccess) {                                                                        \
      (net)->poisoned = true;                                                                      \
      return fail(SDNN_EDEVICE, "%s failed: %s", #call, hipGetErrorString(e_));                   \
    }                                                                                              \
  } while (0)

struct WsLayout {
  size_t act[2], ids[2], src[2], masks[3], rownz, counts, misc, dict, dict16, seglive, part[2], spread, spread_words,
      final_ids, total;
};

// Two activation buffers: row-major [M][N] (path 0) or feature-major tiles of 32 rows (path 1).
WsLayout layout_for(const sdnn_net *net, int64_t M) {
  WsLayout w{};
  const size_t a = 256;
  size_t off = 0;
  const size_t rows = net->path == 1 ? (size_t)((M + 31) / 32) * 32 : (size_t)M;
  const size_t ybytes = align_up(rows * (size_t)net->N * sizeof(float), a);
  w.act[0] = off; off += ybytes;
  w.act[1] = off; off += ybytes;
  const size_t ib = align_up((size_t)std::max<int64_t>(M, 1) * sizeof(int), a);
  w.ids[0] = off; off += ib;
  w.ids[1] = off; off += ib;
  w.src[0] = off; off += ib;
  w.src[1] = off; off += ib;
  for (int i = 0; i < 3; ++i) { w.masks[i] = off; off += ib; }
  w.rownz = off; off += ib;
  w.counts = off; off += align_up((size_t)(net->L + 1) * sizeof(int), a);
  w.misc = off; off += a;
  w.dict = off; off += align_up(kDictWords * sizeof(unsigned), a);
  w.dict16 = off;
  if (net->path == 1) off += align_up((size_t)dict_words<2>() * sizeof(unsigned), a);
  w.seglive = off;
  if (net->path == 1) off += align_up(rows / 32 * (size_t)((net->N + 31) / 32) * sizeof(unsigned), a);
  for (int i = 0; i < 2; ++i) {
    w.part[i] = off;
    if (net->path == 1) off += align_up((size_t)kMaxPartWords * sizeof(unsigned), a);
  }
  w.spread = off;
  w.spread_words = net->path == 1 ? rows / 32 * kSpread * kLineWords : 0;
  off += align_up(w.spread_words * sizeof(unsigned), a);
  w.final_ids = off; off += align_up((size_t)std::max<int64_t>(M, 1) * sizeof(long long), a);
  w.total = off;
  return w;
}

sdnn_status check_usable(const sdnn_net *net) {
  if (!net) return fail(SDNN_EINVAL, "null handle");
  if (net->poisoned) return fail(SDNN_EDEVICE, "handle is poisoned by an earlier device error");
  return SDNN_OK;
}

template <int B, int KC>
hipError_t launch_lds(sdnn_net *net, const float *yin, float *yout, const LayerDev &ld, const int *ids,
                      const int *count, int *rownz) {
  static bool configured = false;
  const size_t lds = (size_t)B * net->N * sizeof(float);
  if (!configured) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_layer_lds<B, KC>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsTileBytes);
    if (e != hipSuccess) return e;
    configured = true;
  }
  const int per_cu = lds <= 64 * 1024 ? 2 : 1;
  // distinct columns only, when the layer's duplicates need not be computed
  const bool dd = ld.ell16 && ld.ell16c && ld.cols && ld.dedup_ok;
  const bool placed = !dd && ld.place && ld.pell16;
  hipLaunchKernelGGL((k_layer_lds<B, KC>), dim3(net->cus * per_cu), dim3(1024), lds, net->stream, yin, yout, net->N,
                     ld.ell, ld.K, dd ? ld.ell16c : (placed ? ld.pell16 : ld.ell16), dd ? nullptr : ld.w8, ld.w,
                     ld.bias, net->ymax, ids, count, net->masks, rownz, dd ? ld.cols : nullptr, dd ? ld.D : net->N,
                     placed ? ld.place : nullptr);
  return hipGetLastError();
}

template <int B>
hipError_t launch_lds_k(sdnn_net *net, const float *yin, float *yout, const LayerDev &ld, const int *ids,
                        const int *count, int *rownz) {
  if (ld.K == 32) return launch_lds<B, 32>(net, yin, yout, ld, ids, count, rownz);
  return launch_lds<B, 0>(net, yin, yout, ld, ids, count, rownz);
}

// A layer of at most 8 tiles with K == 32 (see k_layer_gfm_small). Liveness goes to the partial
// words part_out; *S_out and *nt_out receive their slots per tile and tiles.
hipError_t launch_gfm_small(sdnn_net *net, const LayerDev &ld, const float *fin, float *fout, const int *npos,
                            int64_t max_tiles, unsigned *part_out, const unsigned *part_prev, int prev_S, int prev_nt,
                            unsigned *masks_prev, unsigned *masks_clear, int *count_out, const int *live_before,
                            unsigned long long *progress, unsigned long long progress_tag, int *S_out, int *nt_out) {
  const bool dd = ld.src16 && ld.cols && ld.dedup_ok;  // distinct columns only
  const int ncols = dd ? ld.D : net->N;
  const int nchunks = (ncols + 31) / 32;
  const int ntiles_h = (int)std::max<int64_t>(1, std::min<int64_t>(8, max_tiles));
  const int parts = 8 / ntiles_h;
  // at most kMaxPartWords / 8 workgroups per XCD, so that the partial words fit their buffer
  const int per_xcd = std::max(1, std::min({kMaxPartWords / 8, 2 * net->cus, (nchunks + parts - 1) / parts}));
  const dim3 grid(8 * per_xcd);
  *S_out = per_xcd * parts;
  *nt_out = ntiles_h;
  if (ld.uniform && ld.src16)
    hipLaunchKernelGGL((k_layer_gfm_small<32, kWOne>), grid, dim3(kPartThreads), 0, net->stream, fin, fout, net->N,
                       ld.ell, dd ? ld.src16c : ld.src16, (const float *)nullptr, ld.w, ld.bias, net->ymax, npos,
                       ntiles_h, part_out, part_prev, prev_S, prev_nt, masks_prev, masks_clear, count_out, live_before,
                       progress, progress_tag, dd ? ld.cols : nullptr, ncols);
  else if (ld.src16 && ld.w32)
    hipLaunchKernelGGL((k_layer_gfm_small<32, kWEdge>), grid, dim3(kPartThreads), 0, net->stream, fin, fout, net->N,
                       ld.ell, ld.src16, ld.w32, ld.w, ld.bias, net->ymax, npos, ntiles_h, part_out, part_prev, prev_S,
                       prev_nt, masks_prev, masks_clear, count_out, live_before, progress, progress_tag,
                       (const int *)nullptr, net->N);
  else
    hipLaunchKernelGGL((k_layer_gfm_small<32, kWEll>), grid, dim3(kPartThreads), 0, net->stream, fin, fout, net->N,
                       ld.ell, ld.src16, (const float *)nullptr, ld.w, ld.bias, net->ymax, npos, ntiles_h, part_out,
                       part_prev, prev_S, prev_nt, masks_prev, masks_clear, count_out, live_before, progress,
                       progress_tag, (const int *)nullptr, net->N);
  return hipGetLastError();
}

// One layer of the global-tile path: ceil(tiles / 8) launches of 8 tiles each (rounds), reading fin
// and writing fout at the same list positions; *npos is the list length and max_tiles a host bound
// on its tiles. With count_out set (one round only) the launch first counts the previous layer's
// live rows from masks_prev and clears masks_clear.
// Tiles per XCD and launch for a layer that reads `bytes` of each input tile: as many as fit 2 MiB of
// the XCD's 4 MiB L2, at most 8.
int tiles_per_xcd(size_t bytes) {
  return (int)std::max<size_t>(1, std::min<size_t>(8, ((size_t)2 << 20) / std::max<size_t>(bytes, 1)));
}
// Launches of launch_gfm (fp32 tiles) or launch_gfm_u8 (code tiles of cr rows, cr > 0) for a layer
// over max_tiles fp32 tiles.
int32_t gfm_launches(const sdnn_net *net, const LayerDev &ld, int64_t max_tiles, int cr) {
  const bool dd = ld.K == 32 && ld.src16 && ld.cols && ld.dedup_ok;
  const int ncols = dd ? ld.D : net->N;
  if (cr > 0) max_tiles = (max_tiles + cr / 32 - 1) / (cr / 32);
  const int tpx = dd ? tiles_per_xcd((size_t)ncols * (cr > 0 ? cr : 32 * sizeof(float))) : 1;
  return (int32_t)((max_tiles + 8 * tpx - 1) / (8 * tpx));
}

hipError_t launch_gfm(sdnn_net *net, const LayerDev &ld, const float *fin, float *fout, const int *npos,
                      int64_t max_tiles, unsigned *masks, const unsigned *masks_prev = nullptr,
                      unsigned *masks_clear = nullptr, int *count_out = nullptr, unsigned *spread = nullptr) {
  // distinct columns only, when the layer's duplicates need not be computed
  const bool dd = ld.K == 32 && ld.src16 && ld.cols && ld.dedup_ok;
  const int ncols = dd ? ld.D : net->N;
  const int *cols = dd ? ld.cols : nullptr;
  const unsigned short *s16 = dd ? ld.src16c : ld.src16;
  // the few columns of such a layer touch a small part of each tile, so an XCD can keep several
  // tiles in its L2 and a launch covers 8 tpx of them
  const int tpx = dd ? tiles_per_xcd((size_t)ncols * 32 * sizeof(float)) : 1;
  const int rounds = (int)((max_tiles + 8 * tpx - 1) / (8 * tpx));
  // one workgroup per output chunk of a tile's share when the round has fewer than 8 tiles
  const int nchunks = (ncols + kGfmOutputs - 1) / kGfmOutputs;
  const int64_t parts = 8 / std::max<int64_t>(1, std::min<int64_t>(8, max_tiles));
  const int per_xcd = tpx * std::max(1, (int)std::min<int64_t>(net->cus, (nchunks + parts - 1) / parts));
  const dim3 grid(8 * per_xcd);
  for (int r = 0; r < rounds; ++r) {
    int *cnt = r == 0 ? count_out : nullptr;
    if (ld.K == 32 && ld.src16 && ld.uniform)
      hipLaunchKernelGGL((k_layer_gfm<kWOne>), grid, dim3(256), 0, net->stream, fin, fout, net->N, ld.ell, ld.K, s16,
                         (const float *)nullptr, ld.w, ld.bias, net->ymax, npos, masks, r * 8 * tpx, masks_prev,
                         masks_clear, cnt, spread, cols, ncols, tpx);
    else if (ld.K == 32 && ld.src16 && ld.w32)
      hipLaunchKernelGGL((k_layer_gfm<kWEdge>), grid, dim3(256), 0, net->stream, fin, fout, net->N, ld.ell, ld.K,
                         ld.src16, ld.w32, 0.0f, ld.bias, net->ymax, npos, masks, r * 8, masks_prev, masks_clear, cnt,
                         spread, (const int *)nullptr, net->N, 1);
    else
      hipLaunchKernelGGL((k_layer_gfm<kWEll>), grid, dim3(256), 0, net->stream, fin, fout, net->N, ld.ell, ld.K,
                         (const unsigned short *)nullptr, (const float *)nullptr, 0.0f, ld.bias, net->ymax, npos,
                         masks, r * 8, masks_prev, masks_clear, cnt, spread, (const int *)nullptr, net->N, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_to_fm(sdnn_net *net, const float *y, float *fm, const int *ids, const int *count, int *rownz) {
  hipLaunchKernelGGL(k_to_fm<32>, dim3(net->cus * 8), dim3(256), 0, net->stream, y, fm, net->N, ids, count, rownz);
  return hipGetLastError();
}

template <int T>
size_t bits_tile_bytes_needed(const sdnn_net *net) {
  using W = typename BitWord<T>::type;
  return (size_t)net->N * sizeof(W);
}

template <int T>
hipError_t launch_pack_bits(sdnn_net *net, const float *yin, void *bits, const int *ids, const int *count) {
  using W = typename BitWord<T>::type;
  hipLaunchKernelGGL(k_pack_bits<T>, dim3(net->cus * 8), dim3(256), 0, net->stream, yin, reinterpret_cast<W *>(bits),
                     net->N, ids, count, net->rownz, net->misc);
  return hipGetLastError();
}

template <int T, int KC, bool CODES>
hipError_t launch_layer_bits_k(sdnn_net *net, const LayerDev &ld, const void *bits, float *fout, const int *count) {
  using W = typename BitWord<T>::type;
  // one workgroup per CU: 16 waves at up to 128 registers fill the register file; LDS is static
  const int per_cu = 1;
  hipLaunchKernelGGL((k_layer_bits<T, KC, CODES>), dim3(net->cus * per_cu), dim3(kBitsThreads), 0, net->stream,
                     reinterpret_cast<const W *>(bits), fout, net->N, ld.ellw, ld.K, ld.bias, net->ymax,
                     count, net->masks, net->dict, net->misc + kOverflowSlot, net->misc);
  return hipGetLastError();
}

// codes: write one-byte dictionary codes instead of fp32 values
template <int T>
hipError_t launch_layer_bits(sdnn_net *net, const LayerDev &ld, const void *bits, float *fout, const int *count,
                             bool codes) {
  if (codes) {
    if (ld.K == 32) return launch_layer_bits_k<T, 32, true>(net, ld, bits, fout, count);
    return launch_layer_bits_k<T, 0, true>(net, ld, bits, fout, count);
  }
  if (ld.K == 32) return launch_layer_bits_k<T, 32, false>(net, ld, bits, fout, count);
  return launch_layer_bits_k<T, 0, false>(net, ld, bits, fout, count);
}

// Source order for the counting kernel. A wave's LDS read of one source slot serves 64 outputs, in
// two halves of 32 lanes (32 consecutive output positions); within a half, reads of different
// 4-byte words in the same one of the 32 banks are served one after another. The count does not
// depend on the order of a column's sources, so for each half the sources are dealt to the 32
// slots greedily: slot by slot, lanes with the fewest distinct remaining banks choose first, each
// taking a remaining source whose bank this slot has used least. src: [4][D][8] u16 lists; wbytes:
// bytes per LDS word of the bit tile (the word of source k is k * wbytes / 4).
std::vector<uint16_t> bank_balanced_lists(const uint16_t *src, int D, int wbytes) {
  std::vector<uint16_t> out((size_t)32 * D);
  const int groups = (D + 31) / 32;
  parallel_for(groups, [&](int32_t g) {
    const int p0 = g * 32, np = std::min(32, D - p0);
    uint16_t rem[32][32];
    int nrem[32];
    for (int i = 0; i < np; ++i) {
      for (int sl = 0; sl < 32; ++sl) rem[i][sl] = src[((size_t)(sl / 8) * D + p0 + i) * 8 + sl % 8];
      nrem[i] = 32;
    }
    auto word = [&](unsigned k) { return (unsigned)((k * (unsigned)wbytes) / 4u); };
    for (int sl = 0; sl < 32; ++sl) {
      int load[32] = {0};
      unsigned used[32][32];  // words of each bank read in this slot
      int order[32], key[32];
      for (int i = 0; i < np; ++i) {
        unsigned seen = 0u;
        for (int q = 0; q < nrem[i]; ++q) seen |= 1u << (word(rem[i][q]) & 31u);
        key[i] = __builtin_popcount(seen);
        order[i] = i;
      }
      std::stable_sort(order, order + np, [&](int a, int b) { return key[a] < key[b]; });
      for (int oi = 0; oi < np; ++oi) {
        const int i = order[oi];
        int best = 0, bcost = 1 << 30;
        for (int q = 0; q < nrem[i]; ++q) {
          const unsigned w = word(rem[i][q]), b = w & 31u;
          bool same = false;
          for (int u = 0; u < load[b]; ++u) same = same || used[b][u] == w;
          const int cost = same ? 0 : load[b] + 1;
          if (cost < bcost) { bcost = cost; best = q; }
        }
        const uint16_t k = rem[i][best];
        rem[i][best] = rem[i][--nrem[i]];
        const unsigned w = word(k), b = w & 31u;
        bool same = false;
        for (int u = 0; u < load[b]; ++u) same = same || used[b][u] == w;
        if (!same) used[b][load[b]++] = w;
        out[((size_t)(sl / 8) * D + p0 + i) * 8 + sl % 8] = k;
      }
    }
  });
  return out;
}

// Column order for the fused LDS kernel: a wave's 16-byte LDS reads of one source slot are served
// 16 lanes at a time, and reads of different rows in the same 16-byte bank group are served one
// after another. With B-row tiles (B = 4, 8, 16) an output takes B / 4 lanes, so a cycle serves
// G = 64 / B consecutive positions, and row k covers bank groups (B / 4) k .. (B / 4) k + B / 4 - 1
// mod 16: two of the G columns collide when their sources agree mod G. The fp32 chain fixes the
// order of a column's sources, but which columns share a read is free, so positions are filled in
// groups of G: each group starts from a remaining column and repeatedly takes, among 128 sampled
// remaining columns, the one whose sources add the fewest collisions over the 32 slots.
// lists: D x 32 sources by position; returns the positions' new order.
std::vector<int32_t> conflict_grouped_order(const std::vector<uint16_t> &lists, int D, int G) {
  std::vector<int32_t> order, rem((size_t)D);
  order.reserve((size_t)D);
  for (int i = 0; i < D; ++i) rem[(size_t)i] = i;
  uint64_t st = 0x5DEECE66Dull + (uint64_t)D;
  auto next = [&]() {  // SplitMix64
    uint64_t z = (st += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  };
  auto take = [&](size_t idx) {
    const int32_t c = rem[idx];
    rem[idx] = rem.back();
    rem.pop_back();
    return c;
  };
  while (!rem.empty()) {
    uint8_t load[32][16] = {};
    auto add = [&](int32_t c) {
      for (int sl = 0; sl < 32; ++sl) ++load[sl][lists[(size_t)c * 32 + sl] % (unsigned)G];
      order.push_back(c);
    };
    add(take((size_t)(next() % rem.size())));
    for (int g = 1; g < G && !rem.empty(); ++g) {
      size_t best = 0;
      int bcost = 1 << 30;
      for (int t = 0; t < 128; ++t) {
        const size_t idx = (size_t)(next() % rem.size());
        const uint16_t *l = lists.data() + (size_t)rem[idx] * 32;
        int cost = 0;
        for (int sl = 0; sl < 32; ++sl) cost += load[sl][l[sl] % (unsigned)G];
        if (cost < bcost) { bcost = cost; best = idx; }
      }
      add(take(best));
    }
  }
  return order;
}

// Layer 0 of a uniform layer by counting (see k_layer_count): dictionary, then the counts as codes
// (cout) or, with yout set, as fp32 rows yout[ids[p]] (masks: one bit per list position).
template <int T, bool ROWMAJOR>
hipError_t launch_layer_count_k(sdnn_net *net, const LayerDev &ld, const void *bits, unsigned char *cout,
                                const int *count, float *yout, const int *ids, unsigned *masks) {
  using W = typename BitWord<T>::type;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_layer_count<T, ROWMAJOR>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    configured = true;
  }
  hipLaunchKernelGGL(k_count_dict, dim3(1), dim3(64), 0, net->stream, net->dict, net->misc, ld.K, ld.w, ld.b, net->ymax);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  size_t lds = 16 + ((size_t)net->N * sizeof(W) + 15) / 16 * 16;
  if (ROWMAJOR) lds += kDictSlots * sizeof(float) + T * sizeof(int);
  // distinct columns only, when the layer's duplicates need not be computed
  const bool dd = ld.cols && ld.ell16c && ld.dedup_ok;
  hipLaunchKernelGGL((k_layer_count<T, ROWMAJOR>), dim3(net->cus), dim3(1024), lds, net->stream,
                     reinterpret_cast<const W *>(bits), cout, net->N,
                     dd ? (ld.ell16cs ? ld.ell16cs : ld.ell16c) : (ld.ell16s ? ld.ell16s : ld.ell16), net->misc, count, masks,
                     yout, ids, reinterpret_cast<const unsigned *>(net->dict), dd ? ld.cols : nullptr,
                     dd ? ld.D : net->N, net->misc);
  return hipGetLastError();
}
template <int T>
hipError_t launch_layer_count(sdnn_net *net, const LayerDev &ld, const void *bits, unsigned char *cout,
                              const int *count) {
  return launch_layer_count_k<T, false>(net, ld, bits, cout, count, nullptr, nullptr, net->masks);
}

// A layer whose input tiles hold dictionary codes of CR rows (see k_layer_gfm_u8); rounds of 8 code
// tiles. max_tiles: host bound on the 32-row tiles of the list.
template <int CR, int CB = 1>
hipError_t launch_gfm_u8_cr(sdnn_net *net, const LayerDev &ld, const unsigned char *cin, float *fout, const int *npos,
                            int64_t max_tiles, unsigned *masks, bool *seglive_used) {
  max_tiles = (max_tiles + CR / 32 - 1) / (CR / 32);  // code tiles
  // distinct columns only, when the layer's duplicates need not be computed (every segment of them
  // is then stored and seglive is not written)
  const bool dd = ld.K == 32 && ld.src16 && ld.cols && ld.dedup_ok;
  const int ncols = dd ? ld.D : net->N;
  *seglive_used = !dd;
  const int tpx = dd ? tiles_per_xcd((size_t)ncols * CR * CB) : 1;  // see launch_gfm
  const int nchunks = (ncols + u8_outputs(CR) - 1) / u8_outputs(CR);
  const int64_t parts = 8 / std::max<int64_t>(1, std::min<int64_t>(8, max_tiles));
  const int per_xcd = tpx * std::max(1, (int)std::min<int64_t>(net->cus, (nchunks + parts - 1) / parts));
  const dim3 grid(8 * per_xcd);
  const int rounds = (int)((max_tiles + 8 * tpx - 1) / (8 * tpx));
  const float *dict = reinterpret_cast<const float *>(CB == 1 ? net->dict : net->dict16);
  for (int r = 0; r < rounds; ++r) {
    // (two-byte codes come only from encodings, which the opt-in uniform-layer kernels never use)
    if constexpr (CB == 1) {
      if (ld.K == 32 && ld.src16 && ld.uniform) {
        hipLaunchKernelGGL((k_layer_gfm_u8<kWOne, CR, u8_rows_per_lane(CR), u8_outs_per_lane(CR), CB>), grid, dim3(256), 0, net->stream, cin, fout, net->N, ld.ell, ld.K,
                           dd ? ld.src16c : ld.src16, (const float *)nullptr, ld.w, ld.bias, net->ymax, dict, npos, masks,
                           net->seglive, r * 8 * tpx, net->spread, dd ? ld.cols : nullptr, ncols, tpx);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        continue;
      }
    } else if (ld.uniform) {
      return hipErrorInvalidValue;
    }
    if (ld.K == 32 && ld.src16 && ld.w32)
      hipLaunchKernelGGL((k_layer_gfm_u8<kWEdge, CR, u8_rows_per_lane(CR), u8_outs_per_lane(CR), CB>), grid, dim3(256), 0, net->stream, cin, fout, net->N, ld.ell,
                         ld.K, ld.src16, ld.w32, 0.0f, ld.bias, net->ymax, dict, npos, masks, net->seglive, r * 8,
                         net->spread, (const int *)nullptr, net->N, 1);
    else
      hipLaunchKernelGGL((k_layer_gfm_u8<kWEll, CR, u8_rows_per_lane(CR), u8_outs_per_lane(CR), CB>), grid, dim3(256), 0, net->stream, cin, fout, net->N, ld.ell,
                         ld.K, (const unsigned short *)nullptr, (const float *)nullptr, 0.0f, ld.bias, net->ymax, dict,
                         npos, masks, net->seglive, r * 8, net->spread, (const int *)nullptr, net->N, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
hipError_t launch_gfm_u8(sdnn_net *net, const LayerDev &ld, const unsigned char *cin, float *fout, const int *npos,
                         int64_t max_tiles, unsigned *masks, bool *seglive_used) {
  return code_rows(net->bitsT) == 128 ? launch_gfm_u8_cr<128>(net, ld, cin, fout, npos, max_tiles, masks, seglive_used)
                                      : launch_gfm_u8_cr<64>(net, ld, cin, fout, npos, max_tiles, masks, seglive_used);
}
// A layer whose inputs are two-byte codes (64-row code tiles, dictionary dict16; only layers wider
// than 32768 neurons use them, and those have 64-row code tiles)
hipError_t launch_gfm_u16(sdnn_net *net, const LayerDev &ld, const unsigned char *cin, float *fout, const int *npos,
                          int64_t max_tiles, unsigned *masks, bool *seglive_used) {
  if (code_rows(net->bitsT) != 64) return hipErrorInvalidValue;
  return launch_gfm_u8_cr<64, 2>(net, ld, cin, fout, npos, max_tiles, masks, seglive_used);
}

// Rows per workgroup of k_layers_lds: at most the largest of 16, 8, 4 whose two tiles fit 128 KiB
// of LDS, halved (down to 1) while twice the workgroups still fit one per CU.
int fused_rows_max(const sdnn_net *net) {
  int b = 16;
  while (b > 4 && (size_t)2 * b * net->N * sizeof(float) > (size_t)kLdsTileBytes) b /= 2;
  return b;
}
int fused_rows(const sdnn_net *net, int64_t rows) {
  int b = fused_rows_max(net);
  while (b > 1 && 2 * ((rows + b - 1) / b) <= net->cus) b /= 2;
  return b;
}

template <int B>
hipError_t launch_layers_lds_b(sdnn_net *net, const float *yin, float *yout, int l0, const int *ids, const int *count,
                               int64_t rows) {
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_layers_lds<B>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsTileBytes);
    if (e != hipSuccess) return e;
    configured = true;
  }
  int shift = 0;
  while ((1 << shift) < net->B * (int)sizeof(float)) ++shift;
  const size_t lds = (size_t)2 * net->N * B * sizeof(float);
  const int grid = (int)std::max<int64_t>(1, (rows + B - 1) / B);
  const LayerPtr *lp = net->lp_dev[B >= 16 ? 2 : (B == 8 ? 1 : 0)];  // the table grouped for this height
  hipLaunchKernelGGL(k_layers_lds<B>, dim3(grid), dim3(1024), lds, net->stream, yin, yout, net->N, lp, l0,
                     net->L, net->ymax, ids, count, net->counts, net->masks, shift);
  return hipGetLastError();
}

// Layers [l0, L) of at most `rows` live rows (list ids, count *count) in one launch (k_layers_lds).
hipError_t launch_layers_lds(sdnn_net *net, const float *yin, float *yout, int l0, const int *ids, const int *count,
                             int64_t rows) {
  switch (fused_rows(net, rows)) {
    case 16: return launch_layers_lds_b<16>(net, yin, yout, l0, ids, count, rows);
    case 8: return launch_layers_lds_b<8>(net, yin, yout, l0, ids, count, rows);
    case 4: return launch_layers_lds_b<4>(net, yin, yout, l0, ids, count, rows);
    case 2: return launch_layers_lds_b<2>(net, yin, yout, l0, ids, count, rows);
    default: return launch_layers_lds_b<1>(net, yin, yout, l0, ids, count, rows);
  }
}

// One layer of the LDS-tile path.
hipError_t launch_layer(sdnn_net *net, int l, const float *yin, float *yout, const int *ids, const int *count,
                        int *rownz) {
  const LayerDev &ld = net->layers[l];
  switch (net->B) {
    case 32: return launch_lds_k<32>(net, yin, yout, ld, ids, count, rownz);
    case 16: return launch_lds_k<16>(net, yin, yout, ld, ids, count, rownz);
    default: return launch_lds_k<8>(net, yin, yout, ld, ids, count, rownz);
  }
}

}  // namespace

extern "C" {

const char *sdnn_last_error(void) { return g_err.c_str(); }

sdnn_status sdnn_create(sdnn_net **out, int32_t n_neurons, int32_t n_layers, float ymax) {
  if (!out) return fail(SDNN_EINVAL, "out is null");
  *out = nullptr;
  if (n_neurons < 1 || n_neurons > kMaxNeurons) return fail(SDNN_EINVAL, "n_neurons %d not in [1, %d]", n_neurons, kMaxNeurons);
  if (n_layers < 1 || n_layers > kMaxLayers) return fail(SDNN_EINVAL, "n_layers %d not in [1, %d]", n_layers, kMaxLayers);
  if (!std::isfinite(ymax) || !(ymax > 0.0f)) return fail(SDNN_EINVAL, "ymax must be finite and > 0");
  sdnn_net *net = new (std::nothrow) sdnn_net;
  if (!net) return fail(SDNN_ENOMEM, "out of host memory");
  net->N = n_neurons;
  net->L = n_layers;
  net->ymax = ymax;
  net->layers.resize((size_t)n_layers);
  // LDS tile of B rows x N fp32 must fit the budget with B >= 8
  if ((size_t)32 * n_neurons * sizeof(float) <= (size_t)kLdsTileBytes) { net->path = 0; net->B = 32; }
  else if ((size_t)16 * n_neurons * sizeof(float) <= (size_t)kLdsTileBytes) { net->path = 0; net->B = 16; }
  else if ((size_t)8 * n_neurons * sizeof(float) <= (size_t)kLdsTileBytes) { net->path = 0; net->B = 8; }
  else {
    // global feature-major tiles of 32 rows (128-byte segments per source); one tile per XCD per
    // launch, held in that XCD's L2 up to 16384 neurons and in the Infinity Cache beyond
    net->path = 1;
    net->B = 32;
    // layer 0 from bit tiles: 32-row tiles while their words fit 64 KiB of LDS, else 16-row tiles
    net->bitsT = (size_t)n_neurons * 4 <= 64 * 1024 ? 32 : ((size_t)n_neurons * 2 <= 128 * 1024 ? 16 : 0);
  }
  *out = net;
  g_err.clear();
  return SDNN_OK;
}

int32_t sdnn_kernel_path(const sdnn_net *net) { return net ? net->path : -1; }

sdnn_status sdnn_enable_equal_value_kernels(sdnn_net *net, int32_t enable) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (enable != 0 && enable != 1) return fail(SDNN_EINVAL, "enable must be 0 or 1");
  if (net->n_loaded > 0) return fail(SDNN_ESTATE, "layers are already loaded");
  net->equal_value_kernels = enable != 0;
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_load_layers(sdnn_net *net, int32_t l0, int32_t nl, const int64_t *col_ptr, const int32_t *row_idx,
                             const float *val, const float *bias, void *hip_stream) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (nl < 1 || l0 < 0 || (int64_t)l0 + nl > net->L) return fail(SDNN_EINVAL, "layers [%d, %d) outside [0, %d)", l0, l0 + nl, net->L);
  if (!col_ptr || !row_idx || !val || !bias) return fail(SDNN_EINVAL, "null array");
  for (int32_t i = 0; i < nl; ++i)
    if (net->layers[(size_t)l0 + i].ell) return fail(SDNN_ESTATE, "layer %d already loaded", l0 + i);
  const int32_t N = net->N;
  for (int32_t i = 1; i < nl; ++i)
    if (col_ptr[(size_t)i * (N + 1)] != col_ptr[(size_t)(i - 1) * (N + 1) + N])
      return fail(SDNN_EINVAL, "layer %d does not start where layer %d ends", l0 + i, l0 + i - 1);
  if (col_ptr[0] < 0) return fail(SDNN_EINVAL, "negative column offset");
  // ---- validate every layer before touching the device (layers in parallel on host threads)
  std::vector<int> K((size_t)nl, 0);
  std::vector<char> uniform((size_t)nl, 0);
  std::vector<std::string> err((size_t)nl);
  parallel_for(nl, [&](int32_t i) {
    const int64_t *cp = col_ptr + (size_t)i * (N + 1);
    char buf[256];
    int kmax = 0, kmin = kMaxDegree + 1;
    bool same_w = true;
    const int64_t e0 = cp[0];
    for (int32_t j = 0; j < N; ++j) {
      const int64_t a = cp[j], b = cp[j + 1];
      if (b < a) { snprintf(buf, sizeof buf, "layer %d column %d: decreasing offsets", l0 + i, j); err[(size_t)i] = buf; return; }
      if (b - a > kMaxDegree) { snprintf(buf, sizeof buf, "layer %d column %d: %lld sources exceed %d", l0 + i, j, (long long)(b - a), kMaxDegree); err[(size_t)i] = buf; return; }
      for (int64_t e = a; e < b; ++e) {
        const int32_t k = row_idx[e];
        if (k < 0 || k >= N) { snprintf(buf, sizeof buf, "layer %d column %d: source %d out of range", l0 + i, j, k); err[(size_t)i] = buf; return; }
        if (e > a && k <= row_idx[e - 1]) { snprintf(buf, sizeof buf, "layer %d column %d: sources not strictly ascending", l0 + i, j); err[(size_t)i] = buf; return; }
        if (!std::isfinite(val[e])) { snprintf(buf, sizeof buf, "layer %d column %d: non-finite weight", l0 + i, j); err[(size_t)i] = buf; return; }
        same_w = same_w && std::memcmp(&val[e], &val[e0], sizeof(float)) == 0;
      }
      kmax = std::max<int>(kmax, (int)(b - a));
      kmin = std::min<int>(kmin, (int)(b - a));
    }
    bool same_b = true;
    for (int32_t j = 0; j < N; ++j) {
      if (!std::isfinite(bias[(size_t)i * N + j])) { snprintf(buf, sizeof buf, "layer %d: non-finite bias", l0 + i); err[(size_t)i] = buf; return; }
      same_b = same_b && std::memcmp(&bias[(size_t)i * N + j], &bias[(size_t)i * N], sizeof(float)) == 0;
    }
    K[(size_t)i] = std::max(kmax, 1);
    // the specialisations that read one weight and one bias per layer are opt-in: by default every
    // layer reads each edge's weight and each neuron's bias from memory, whatever their values
    uniform[(size_t)i] = net->equal_value_kernels && kmax > 0 && kmin == kmax && same_w && same_b;
  });
  for (int32_t i = 0; i < nl; ++i)
    if (!err[(size_t)i].empty()) return fail(SDNN_EINVAL, "%s", err[(size_t)i].c_str());
  // ---- duplicate columns (uniform layers with 32 sources per column): columns
  // with the same source list have the same output, so reps[i][j] = the smallest column with j's
  // list (empty: no duplicates). Grouping uses the sources as given; equal lists stay equal once
  // mapped (below). With the Kronecker-expanded networks of Sec. III every 16 columns of a block
  // share their list.
  std::vector<std::vector<int32_t>> reps((size_t)nl);
  parallel_for(nl, [&](int32_t i) {
    if (N > 65536 || !uniform[(size_t)i] || K[(size_t)i] != 32) return;
    const int64_t *cp = col_ptr + (size_t)i * (N + 1);
    std::unordered_map<uint64_t, std::vector<int32_t>> seen;
    seen.reserve((size_t)N);
    std::vector<int32_t> r((size_t)N);
    int32_t distinct = 0;
    for (int32_t j = 0; j < N; ++j) {
      const int32_t *src = row_idx + cp[j];
      uint64_t h = 0x9E3779B97F4A7C15ull;
      for (int k = 0; k < 32; ++k) {
        h ^= (uint32_t)src[k] + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
        h *= 0xBF58476D1CE4E5B9ull;
      }
      std::vector<int32_t> &cand = seen[h];
      int32_t found = -1;
      for (int32_t c : cand)
        if (std::memcmp(row_idx + cp[c], src, 32 * sizeof(int32_t)) == 0) { found = c; break; }
      if (found < 0) {
        cand.push_back(j);
        found = j;
        ++distinct;
      }
      r[(size_t)j] = found;
    }
    if (distinct < N) reps[(size_t)i] = std::move(r);
  });
  // ---- a layer loaded right after one with duplicates reads that layer's representatives only:
  // its sources are mapped through them (values are equal), and the earlier layer may then skip
  // its duplicate columns. mapped[i] holds layer i's mapped sources (empty: as given).
  std::vector<std::vector<int32_t>> mapped((size_t)nl);
  std::vector<char> maps_prev((size_t)nl, 0);  // layer l0 + i's sources go through layer l0 + i - 1's reps
  {
    const std::vector<int32_t> *prev = (net->prev_rep_layer == l0 - 1 && !net->prev_rep.empty()) ? &net->prev_rep : nullptr;
    for (int32_t i = 0; i < nl; ++i) {
      if (prev) {
        const int64_t *cp = col_ptr + (size_t)i * (N + 1);
        const int64_t e0 = cp[0], e1 = cp[N];
        std::vector<int32_t> &m = mapped[(size_t)i];
        m.resize((size_t)(e1 - e0));
        for (int64_t e = e0; e < e1; ++e) m[(size_t)(e - e0)] = (*prev)[(size_t)row_idx[e]];
        maps_prev[(size_t)i] = 1;
      }
      prev = reps[(size_t)i].empty() ? nullptr : &reps[(size_t)i];
    }
  }
  // source of entry e of layer i (absolute index into row_idx)
  auto src_at = [&](int32_t i, int64_t e) -> int32_t {
    const std::vector<int32_t> &m = mapped[(size_t)i];
    return m.empty() ? row_idx[e] : m[(size_t)(e - col_ptr[(size_t)i * (N + 1)])];
  };
  // ---- pack: slot-major ELL [K][N] of (byte offset of source row in the tile, weight bits)
  const int stride = net->B * (int)sizeof(float);
  std::vector<size_t> layer_off((size_t)nl + 1, 0);
  for (int32_t i = 0; i < nl; ++i) layer_off[(size_t)i + 1] = layer_off[(size_t)i] + (size_t)N * K[(size_t)i];
  const size_t ell_words = layer_off[(size_t)nl];
  const size_t ell_bytes = align_up(ell_words * sizeof(int2), 256);
  const size_t bias_bytes = (size_t)nl * N * sizeof(float);
  std::vector<int2> host_ell;
  try {
    host_ell.resize(ell_words);
  } catch (...) {
    return fail(SDNN_ENOMEM, "out of host memory packing %zu bytes", ell_words * sizeof(int2));
  }
  parallel_for(nl, [&](int32_t i) {
    const int64_t *cp = col_ptr + (size_t)i * (N + 1);
    const int Ki = K[(size_t)i];
    int2 *base = host_ell.data() + layer_off[(size_t)i];
    for (int32_t j = 0; j < N; ++j) {
      int s = 0;
      for (int64_t e = cp[j]; e < cp[j + 1]; ++e, ++s) {
        int wbits;
        std::memcpy(&wbits, &val[e], sizeof(int));
        base[(size_t)s * N + j] = make_int2(src_at(i, e) * stride, wbits);
      }
      for (; s < Ki; ++s) base[(size_t)s * N + j] = make_int2(0, 0);
    }
  });
  // ---- device copy
  if (net->device < 0) {
    HIP_OR_POISON(net, hipGetDevice(&net->device));
    HIP_OR_POISON(net, hipDeviceGetAttribute(&net->cus, hipDeviceAttributeMultiprocessorCount, net->device));
    // the host-side objects sdnn_infer uses (read-back events, pinned read-back slots, the progress
    // word in coherent host memory), created once here so that the timed calls allocate nothing
    net->events.resize(4);
    for (auto &ev : net->events) HIP_OR_POISON(net, hipEventCreateWithFlags(&ev, hipEventDisableTiming));
    HIP_OR_POISON(net, hipHostMalloc(reinterpret_cast<void **>(&net->pinned), 8 * sizeof(int32_t), hipHostMallocDefault));
    HIP_OR_POISON(net, hipHostMalloc(reinterpret_cast<void **>(&net->progress), sizeof(unsigned long long),
                                     hipHostMallocCoherent));
    *net->progress = 0ull;
    HIP_OR_POISON(net, hipHostGetDevicePointer(reinterpret_cast<void **>(&net->progress_dev), net->progress, 0));
    HIP_OR_POISON(net, hipHostMalloc(reinterpret_cast<void **>(&net->notify), sizeof(unsigned long long),
                                     hipHostMallocCoherent));
    *net->notify = 0ull;
    HIP_OR_POISON(net, hipHostGetDevicePointer(reinterpret_cast<void **>(&net->notify_dev), net->notify, 0));
    // the device address of the static workspace on this device (sdnn_infer_static)
    void *sw = nullptr;
    st = scratch_address(net->device, &sw);
    if (st != SDNN_OK) return st;
  } else {
    int dev = -1;
    HIP_OR_POISON(net, hipGetDevice(&dev));
    if (dev != net->device) return fail(SDNN_EINVAL, "current device %d differs from the handle's device %d", dev, net->device);
  }
  char *mem = nullptr;
  hipError_t e = hipMalloc(reinterpret_cast<void **>(&mem), ell_bytes + bias_bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", ell_bytes + bias_bytes, hipGetErrorString(e));
  }
  net->allocations.push_back(mem);
  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  if (l0 == 0 && net->bitsT > 0 && K[0] <= 32) {
    // layer 0 on the bit route: its ELL again, with source offsets in bit-tile words (k * 128 bytes
    // in a 32-row fp32 tile becomes k * sizeof(word))
    const size_t n0 = (size_t)N * K[0];
    const int wsz = net->bitsT == 32 ? 4 : 2;
    std::vector<int2> hw0(n0);
    for (size_t q = 0; q < n0; ++q) hw0[q] = make_int2(host_ell[q].x / stride * wsz, host_ell[q].y);
    char *m0 = nullptr;
    e = hipMalloc(reinterpret_cast<void **>(&m0), std::max<size_t>(n0, 1) * sizeof(int2));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", n0 * sizeof(int2), hipGetErrorString(e));
    }
    net->allocations.push_back(m0);
    HIP_OR_POISON(net, hipMemcpy(m0, hw0.data(), n0 * sizeof(int2), hipMemcpyHostToDevice));
    net->layers[0].ellw = reinterpret_cast<const int2 *>(m0);
  }
  HIP_OR_POISON(net, hipMemcpyAsync(mem, host_ell.data(), ell_words * sizeof(int2), hipMemcpyHostToDevice, s));
  HIP_OR_POISON(net, hipMemcpyAsync(mem + ell_bytes, bias, bias_bytes, hipMemcpyHostToDevice, s));
  HIP_OR_POISON(net, hipStreamSynchronize(s));
  for (int32_t i = 0; i < nl; ++i) {
    LayerDev &ld = net->layers[(size_t)l0 + i];
    ld.ell = reinterpret_cast<const int2 *>(mem) + layer_off[(size_t)i];
    ld.bias = reinterpret_cast<const float *>(mem + ell_bytes) + (size_t)i * N;
    ld.K = K[(size_t)i];
    ld.uniform = uniform[(size_t)i] != 0;
    if (ld.uniform) {
      ld.w = val[col_ptr[(size_t)i * (N + 1)]];
      ld.b = bias[(size_t)i * N];
    }
  }
  if (net->path == 1 && N <= 65536) {
    // layers with 32 sources per column: 16-bit source lists, [K][N] like the ELL, and unless the
    // layer is uniform its weights [K][N] fp32 (6 bytes per edge for the large-layer kernels)
    std::vector<int32_t> sel;
    for (int32_t i = 0; i < nl; ++i)
      if (net->layers[(size_t)l0 + i].K == 32) sel.push_back(i);
    if (!sel.empty()) {
      const size_t per = (size_t)32 * N;
      std::vector<size_t> woff(sel.size() + 1, 0);  // weight arrays of the non-uniform layers
      for (size_t q = 0; q < sel.size(); ++q)
        woff[q + 1] = woff[q] + (net->layers[(size_t)l0 + sel[q]].uniform ? 0 : per);
      std::vector<uint16_t> hs(per * sel.size());
      std::vector<float> hw(woff[sel.size()]);
      parallel_for((int32_t)sel.size(), [&](int32_t q) {
        const int64_t *cp = col_ptr + (size_t)sel[(size_t)q] * (N + 1);
        uint16_t *dst = hs.data() + per * (size_t)q;
        const bool weights = woff[(size_t)q + 1] > woff[(size_t)q];
        float *wd = hw.data() + woff[(size_t)q];
        for (int32_t j = 0; j < N; ++j) {
          // a column with fewer than 32 sources is padded with (source 0, weight +0), which adds
          // fma(y, +0, acc) = acc exactly, as in the ELL
          const int deg = (int)(cp[j + 1] - cp[j]);
          for (int sl = 0; sl < 32; ++sl) {
            dst[(size_t)sl * N + j] = sl < deg ? (uint16_t)src_at(sel[(size_t)q], cp[j] + sl) : (uint16_t)0;
            if (weights) wd[(size_t)sl * N + j] = sl < deg ? val[cp[j] + sl] : 0.0f;
          }
        }
      });
      const size_t sbytes = align_up(hs.size() * sizeof(uint16_t), 256);
      const size_t wbytes = hw.size() * sizeof(float);
      char *ms = nullptr;
      e = hipMalloc(reinterpret_cast<void **>(&ms), sbytes + wbytes);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", sbytes + wbytes, hipGetErrorString(e));
      }
      net->allocations.push_back(ms);
      HIP_OR_POISON(net, hipMemcpyAsync(ms, hs.data(), hs.size() * sizeof(uint16_t), hipMemcpyHostToDevice, s));
      if (wbytes) HIP_OR_POISON(net, hipMemcpyAsync(ms + sbytes, hw.data(), wbytes, hipMemcpyHostToDevice, s));
      HIP_OR_POISON(net, hipStreamSynchronize(s));
      for (size_t q = 0; q < sel.size(); ++q) {
        LayerDev &ld = net->layers[(size_t)l0 + sel[q]];
        ld.src16 = reinterpret_cast<const unsigned short *>(ms) + per * q;
        if (!ld.uniform) ld.w32 = reinterpret_cast<const float *>(ms + sbytes) + woff[q];
      }
    }
  }
  {
    // 16-bit source indices in groups of 8 per output ([4][N][8] u16, one 16-byte load per group):
    // every layer with 32 sources per column on widths staged in LDS, with its weights grouped the
    // same way ([4][N][8] fp32) unless it is uniform; and layer 0 of a uniform network of any width
    // (for the counting kernel). Columns with fewer than 32 sources are padded with (source 0,
    // weight +0), a no-op term as in the ELL.
    std::vector<int32_t> sel;
    for (int32_t i = 0; i < nl; ++i) {
      const LayerDev &ld = net->layers[(size_t)l0 + i];
      if (ld.K == 32 && N <= 65536 && (net->path == 0 || (ld.uniform && l0 + i == 0))) sel.push_back(i);
    }
    if (!sel.empty()) {
      const size_t per = (size_t)32 * N;
      std::vector<size_t> woff(sel.size() + 1, 0);
      for (size_t q = 0; q < sel.size(); ++q)
        woff[q + 1] = woff[q] + (net->layers[(size_t)l0 + sel[q]].uniform ? 0 : per);
      std::vector<uint16_t> h16(per * sel.size());
      std::vector<float> hw(woff[sel.size()]);
      parallel_for((int32_t)sel.size(), [&](int32_t q) {
        const int64_t *cp = col_ptr + (size_t)sel[(size_t)q] * (N + 1);
        uint16_t *dst = h16.data() + per * (size_t)q;
        const bool weights = woff[(size_t)q + 1] > woff[(size_t)q];
        float *wd = hw.data() + woff[(size_t)q];
        for (int32_t j = 0; j < N; ++j) {
          const int deg = (int)(cp[j + 1] - cp[j]);
          for (int sl = 0; sl < 32; ++sl) {
            const size_t at = ((size_t)(sl / 8) * N + j) * 8 + sl % 8;
            dst[at] = sl < deg ? (uint16_t)src_at(sel[(size_t)q], cp[j] + sl) : (uint16_t)0;
            if (weights) wd[at] = sl < deg ? val[cp[j] + sl] : 0.0f;
          }
        }
      });
      const size_t sbytes = align_up(h16.size() * sizeof(uint16_t), 256);
      const size_t wbytes = hw.size() * sizeof(float);
      char *m16 = nullptr;
      e = hipMalloc(reinterpret_cast<void **>(&m16), sbytes + wbytes);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", sbytes + wbytes, hipGetErrorString(e));
      }
      net->allocations.push_back(m16);
      HIP_OR_POISON(net, hipMemcpy(m16, h16.data(), h16.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      if (wbytes) HIP_OR_POISON(net, hipMemcpy(m16 + sbytes, hw.data(), wbytes, hipMemcpyHostToDevice));
      for (size_t q = 0; q < sel.size(); ++q) {
        LayerDev &ld = net->layers[(size_t)l0 + sel[q]];
        ld.ell16 = reinterpret_cast<const uint4 *>(m16) + (per / 8) * q;
        if (!ld.uniform) ld.w8 = reinterpret_cast<const float *>(m16 + sbytes) + woff[q];
      }
      // LDS row placements of the first layers on widths staged in LDS (bank_placement): per layer
      // place [N] u16 and the placed sources [4][N][8] u16
      std::vector<int32_t> psel;
      for (size_t q = 0; q < sel.size(); ++q)
        if (net->path == 0 && l0 + sel[q] < kPlacedLayers) psel.push_back((int32_t)q);
      if (!psel.empty()) {
        const size_t pbytes = align_up((size_t)N * sizeof(uint16_t), 256);
        const size_t per_layer = pbytes + per * sizeof(uint16_t);
        std::vector<uint16_t> hp(per_layer / sizeof(uint16_t) * psel.size());
        parallel_for((int32_t)psel.size(), [&](int32_t i) {
          const size_t q = (size_t)psel[(size_t)i];
          const uint16_t *src = h16.data() + per * q;
          const std::vector<uint16_t> place =
              bank_placement(src, N, net->B, 0x5DB1ull * (uint64_t)(l0 + sel[q] + 1), 25 * N);
          uint16_t *out = hp.data() + per_layer / sizeof(uint16_t) * (size_t)i;
          std::copy(place.begin(), place.end(), out);
          uint16_t *po = out + pbytes / sizeof(uint16_t);
          for (size_t t = 0; t < per; ++t) po[t] = place[src[t]];
        });
        char *mp = nullptr;
        e = hipMalloc(reinterpret_cast<void **>(&mp), hp.size() * sizeof(uint16_t));
        if (e != hipSuccess) {
          (void)hipGetLastError();
          return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", hp.size() * sizeof(uint16_t),
                      hipGetErrorString(e));
        }
        net->allocations.push_back(mp);
        HIP_OR_POISON(net, hipMemcpy(mp, hp.data(), hp.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
        for (size_t i = 0; i < psel.size(); ++i) {
          LayerDev &ld = net->layers[(size_t)l0 + sel[(size_t)psel[i]]];
          ld.place = reinterpret_cast<const unsigned short *>(mp + per_layer * i);
          ld.pell16 = reinterpret_cast<const uint4 *>(mp + per_layer * i + pbytes);
        }
      }
    }
  }
  {
    // distinct columns: the representatives and their (mapped) source lists, as [32][D] u16 for the
    // global-tile kernels and as [4][D][8] u16 for the LDS-tile and counting kernels
    std::vector<int32_t> sel;
    for (int32_t i = 0; i < nl; ++i) {
      const LayerDev &ld = net->layers[(size_t)l0 + i];
      if (!reps[(size_t)i].empty() && (ld.src16 || ld.ell16)) sel.push_back(i);
    }
    if (!sel.empty()) {
      std::vector<size_t> off(sel.size() + 1, 0);  // in columns
      std::vector<std::vector<int32_t>> cols(sel.size());
      for (size_t q = 0; q < sel.size(); ++q) {
        const std::vector<int32_t> &r = reps[(size_t)sel[q]];
        for (int32_t j = 0; j < N; ++j)
          if (r[(size_t)j] == j) cols[q].push_back(j);
        off[q + 1] = off[q] + cols[q].size();
      }
      const size_t tot = off[sel.size()];
      std::vector<int32_t> hc(tot);
      std::vector<uint16_t> hs((size_t)32 * tot), hg((size_t)32 * tot);
      parallel_for((int32_t)sel.size(), [&](int32_t q) {
        const int64_t *cp = col_ptr + (size_t)sel[(size_t)q] * (N + 1);
        const size_t D = cols[(size_t)q].size();
        uint16_t *ds = hs.data() + (size_t)32 * off[(size_t)q];
        uint16_t *dg = hg.data() + (size_t)32 * off[(size_t)q];
        for (size_t p = 0; p < D; ++p) {
          const int32_t j = cols[(size_t)q][p];
          hc[off[(size_t)q] + p] = j;
          for (int sl = 0; sl < 32; ++sl) {
            const uint16_t v = (uint16_t)src_at(sel[(size_t)q], cp[j] + sl);
            ds[(size_t)sl * D + p] = v;
            dg[((size_t)(sl / 8) * D + p) * 8 + sl % 8] = v;
          }
        }
      });
      const size_t cbytes = align_up(tot * sizeof(int32_t), 256);
      const size_t sbytes = align_up(hs.size() * sizeof(uint16_t), 256);
      char *mc = nullptr;
      e = hipMalloc(reinterpret_cast<void **>(&mc), cbytes + 2 * sbytes);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", cbytes + 2 * sbytes, hipGetErrorString(e));
      }
      net->allocations.push_back(mc);
      HIP_OR_POISON(net, hipMemcpy(mc, hc.data(), tot * sizeof(int32_t), hipMemcpyHostToDevice));
      HIP_OR_POISON(net, hipMemcpy(mc + cbytes, hs.data(), hs.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      HIP_OR_POISON(net, hipMemcpy(mc + cbytes + sbytes, hg.data(), hg.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      for (size_t q = 0; q < sel.size(); ++q) {
        LayerDev &ld = net->layers[(size_t)l0 + sel[q]];
        ld.cols = reinterpret_cast<const int *>(mc) + off[q];
        ld.src16c = ld.src16 ? reinterpret_cast<const unsigned short *>(mc + cbytes) + (size_t)32 * off[q] : nullptr;
        ld.ell16c = ld.ell16 ? reinterpret_cast<const uint4 *>(mc + cbytes + sbytes) + (size_t)4 * off[q] : nullptr;
        ld.D = (int)cols[q].size();
      }
    }
    // layer 0: the lists in the counting kernel's order (words of 4 bytes on the LDS-tile path, of
    // bitsT / 8 bytes on the global-tile path)
    if (l0 == 0 && net->layers[0].ell16 && net->layers[0].w > 0.0f) {
      LayerDev &ld = net->layers[0];
      const int wbytes = net->path == 0 ? 4 : std::max(net->bitsT, 16) / 8;
      const int64_t *cp = col_ptr;
      std::vector<int32_t> c0;
      if (ld.cols)
        for (int32_t j = 0; j < N; ++j)
          if (reps[0][(size_t)j] == j) c0.push_back(j);
      std::vector<uint16_t> full((size_t)32 * N), part((size_t)32 * c0.size());
      for (int32_t j = 0; j < N; ++j)
        for (int sl = 0; sl < 32; ++sl) full[((size_t)(sl / 8) * N + j) * 8 + sl % 8] = (uint16_t)src_at(0, cp[j] + sl);
      const int D0 = (int)c0.size();
      for (int p = 0; p < D0; ++p)
        for (int sl = 0; sl < 32; ++sl)
          part[((size_t)(sl / 8) * D0 + p) * 8 + sl % 8] = (uint16_t)src_at(0, cp[c0[(size_t)p]] + sl);
      const std::vector<uint16_t> bf = bank_balanced_lists(full.data(), N, wbytes);
      const std::vector<uint16_t> bp = D0 ? bank_balanced_lists(part.data(), D0, wbytes) : std::vector<uint16_t>();
      const size_t fb = align_up(bf.size() * sizeof(uint16_t), 256);
      char *mb = nullptr;
      e = hipMalloc(reinterpret_cast<void **>(&mb), fb + bp.size() * sizeof(uint16_t));
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", fb + bp.size() * sizeof(uint16_t), hipGetErrorString(e));
      }
      net->allocations.push_back(mb);
      HIP_OR_POISON(net, hipMemcpy(mb, bf.data(), bf.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      if (D0) HIP_OR_POISON(net, hipMemcpy(mb + fb, bp.data(), bp.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      ld.ell16s = reinterpret_cast<const uint4 *>(mb);
      ld.ell16cs = D0 ? reinterpret_cast<const uint4 *>(mb + fb) : nullptr;
    }
    // widths staged in LDS: positions in groups for the fused kernel, over all columns and over the
    // distinct columns
    if (net->path == 0) {
      // one order per fused tile-height class the width allows (4 << c rows)
      int nclass = 1;
      while (nclass < 3 && (4 << nclass) <= fused_rows_max(net)) ++nclass;
      std::vector<int32_t> gsel;
      for (int32_t i = 0; i < nl; ++i)
        if (net->layers[(size_t)l0 + i].ell16) gsel.push_back(i);
      const size_t ng = gsel.size() * (size_t)nclass;
      // u = (q * nclass + c) * 2 + v: layer gsel[q], class c, v = 0 all columns / 1 distinct ones
      std::vector<std::vector<int32_t>> gcol(2 * ng);
      std::vector<std::vector<uint16_t>> gl(2 * ng);    // their [4][D][8] lists
      std::vector<std::vector<float>> gw(2 * ng);       // and weights (layers with w8)
      parallel_for((int32_t)(2 * ng), [&](int32_t u) {
        const int32_t i = gsel[(size_t)u / 2 / (size_t)nclass];
        const int cls = (u / 2) % nclass;
        const LayerDev &ld = net->layers[(size_t)l0 + i];
        std::vector<int32_t> pos;
        if (u % 2 == 0) {
          pos.resize((size_t)N);
          for (int32_t j = 0; j < N; ++j) pos[(size_t)j] = j;
        } else if (ld.cols) {
          for (int32_t j = 0; j < N; ++j)
            if (reps[(size_t)i][(size_t)j] == j) pos.push_back(j);
        }
        if (pos.empty()) return;
        const int64_t *cp = col_ptr + (size_t)i * (N + 1);
        const int D = (int)pos.size();
        const bool weights = ld.w8 != nullptr;
        // sources (and weights) by position; short columns padded with (0, +0) as in ell16
        std::vector<uint16_t> lists((size_t)D * 32);
        std::vector<float> wl(weights ? (size_t)D * 32 : 0);
        for (int p = 0; p < D; ++p) {
          const int32_t j = pos[(size_t)p];
          const int deg = (int)(cp[j + 1] - cp[j]);
          for (int sl = 0; sl < 32; ++sl) {
            lists[(size_t)p * 32 + sl] = sl < deg ? (uint16_t)src_at(i, cp[j] + sl) : (uint16_t)0;
            if (weights) wl[(size_t)p * 32 + sl] = sl < deg ? val[cp[j] + sl] : 0.0f;
          }
        }
        const std::vector<int32_t> ord = conflict_grouped_order(lists, D, 16 >> cls);
        std::vector<int32_t> &gc = gcol[(size_t)u];
        std::vector<uint16_t> &g16 = gl[(size_t)u];
        std::vector<float> &g32 = gw[(size_t)u];
        gc.resize((size_t)D);
        g16.resize((size_t)D * 32);
        if (weights) g32.resize((size_t)D * 32);
        for (int p = 0; p < D; ++p) {
          const int32_t q = ord[(size_t)p];
          gc[(size_t)p] = pos[(size_t)q];
          for (int sl = 0; sl < 32; ++sl) {
            const size_t at = ((size_t)(sl / 8) * D + p) * 8 + sl % 8;
            g16[at] = lists[(size_t)q * 32 + sl];
            if (weights) g32[at] = wl[(size_t)q * 32 + sl];
          }
        }
      });
      size_t bytes = 0;
      std::vector<size_t> co(2 * ng), lo(2 * ng), wo(2 * ng);
      for (size_t u = 0; u < 2 * ng; ++u) {
        co[u] = bytes;
        bytes += align_up(gcol[u].size() * sizeof(int32_t), 256);
        lo[u] = bytes;
        bytes += align_up(gl[u].size() * sizeof(uint16_t), 256);
        wo[u] = bytes;
        bytes += align_up(gw[u].size() * sizeof(float), 256);
      }
      if (bytes) {
        char *mg = nullptr;
        e = hipMalloc(reinterpret_cast<void **>(&mg), bytes);
        if (e != hipSuccess) {
          (void)hipGetLastError();
          return fail(SDNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", bytes, hipGetErrorString(e));
        }
        net->allocations.push_back(mg);
        for (size_t u = 0; u < 2 * ng; ++u) {
          if (gcol[u].empty()) continue;
          HIP_OR_POISON(net, hipMemcpy(mg + co[u], gcol[u].data(), gcol[u].size() * sizeof(int32_t), hipMemcpyHostToDevice));
          HIP_OR_POISON(net, hipMemcpy(mg + lo[u], gl[u].data(), gl[u].size() * sizeof(uint16_t), hipMemcpyHostToDevice));
          if (!gw[u].empty())
            HIP_OR_POISON(net, hipMemcpy(mg + wo[u], gw[u].data(), gw[u].size() * sizeof(float), hipMemcpyHostToDevice));
          LayerDev &ld = net->layers[(size_t)l0 + gsel[u / 2 / (size_t)nclass]];
          const int cls = (int)((u / 2) % (size_t)nclass);
          const int *gc = reinterpret_cast<const int *>(mg + co[u]);
          const uint4 *g16 = reinterpret_cast<const uint4 *>(mg + lo[u]);
          if (u % 2 == 0) {
            ld.gcols[cls] = gc;
            ld.gell16[cls] = g16;
            if (!gw[u].empty()) ld.gw8[cls] = reinterpret_cast<const float *>(mg + wo[u]);
          }
          else { ld.gcolsc[cls] = gc; ld.gell16c[cls] = g16; }
        }
      }
    }
    // a layer whose successor reads its representatives only may skip its duplicates; so may the
    // last layer (the final rows are expanded through its representatives)
    for (int32_t i = 0; i < nl; ++i) {
      if (maps_prev[(size_t)i]) net->layers[(size_t)l0 + i - 1].dedup_ok = true;
      if (l0 + i == net->L - 1 && !reps[(size_t)i].empty()) {
        net->layers[(size_t)l0 + i].dedup_ok = true;
        net->last_rep = reps[(size_t)i];
      }
    }
    net->prev_rep = std::move(reps[(size_t)nl - 1]);
    net->prev_rep_layer = net->prev_rep.empty() ? -1 : l0 + nl - 1;
  }
  // the device tables of layers (for launches that run several layers), one per tile-height class
  if (!net->lp_dev[0]) {
    LayerPtr *t = nullptr;
    e = hipMalloc(reinterpret_cast<void **>(&t), (size_t)3 * net->L * sizeof(LayerPtr));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(SDNN_ENOMEM, "hipMalloc of the layer table failed: %s", hipGetErrorString(e));
    }
    net->allocations.push_back(t);
    for (int c = 0; c < 3; ++c) net->lp_dev[c] = t + (size_t)c * net->L;
  }
  {
    // from layer l0 - 1 when this load let it skip its duplicate columns
    const int32_t t0 = (l0 > 0 && net->layers[(size_t)l0 - 1].dedup_ok) ? l0 - 1 : l0;
    std::vector<LayerPtr> hp((size_t)(l0 + nl - t0));
    for (int c = 0; c < 3; ++c) {
      for (int32_t l = t0; l < l0 + nl; ++l) {
        const LayerDev &ld = net->layers[(size_t)l];
        const bool dd = ld.ell16 && ld.ell16c && ld.cols && ld.dedup_ok;
        // the fused kernel reads the positions in their grouped order where there is one
        const uint4 *g16 = dd ? ld.gell16c[c] : ld.gell16[c];
        const uint4 *e16 = g16 ? g16 : (dd ? ld.ell16c : ld.ell16);
        const int *cl = g16 ? (dd ? ld.gcolsc[c] : ld.gcols[c]) : (dd ? ld.cols : nullptr);
        // per-edge weights in the same grouping as the sources (null for a uniform layer)
        const float *w8 = ld.w8 ? (g16 ? ld.gw8[c] : ld.w8) : nullptr;
        hp[(size_t)(l - t0)] = LayerPtr{ld.ell, e16, w8, ld.bias, cl, ld.w, ld.K, dd ? ld.D : N};
      }
      HIP_OR_POISON(net, hipMemcpy(net->lp_dev[c] + t0, hp.data(), hp.size() * sizeof(LayerPtr), hipMemcpyHostToDevice));
    }
  }
  net->n_loaded += nl;
  g_err.clear();
  return SDNN_OK;
}

size_t sdnn_workspace_bytes(const sdnn_net *net, int64_t n_rows) {
  if (!net || n_rows < 0) return 0;
  return layout_for(net, n_rows).total;
}

namespace {

// Read-back ring for the live count: every kPollEvery layers the count is copied to pinned host
// memory behind an event; the host checks it two chunks later, so the stream never drains while
// the host waits.
struct PollRing {
  int slot[4], bound[4], n = 0, head = 0, next = 0;
};

// After layer l (every kPollEvery layers), enqueue a poll of counts[idx], a live count known once
// layer l has finished, and consume polls that are two chunks old. *live_bound receives the
// smallest count seen.
hipError_t poll_step(sdnn_net *net, PollRing &ring, int32_t l, int32_t idx, int64_t *live_bound) {
  hipStream_t s = net->stream;
  if ((l + 1) % kPollEvery != 0 || l + 1 >= net->L) return hipSuccess;
  const int slot = ring.next;
  ring.next = (ring.next + 1) % 4;
  hipError_t e = hipMemcpyAsync(net->pinned + slot, net->counts + idx, sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  e = hipEventRecord(net->events[(size_t)slot], s);
  if (e != hipSuccess) return e;
  ring.slot[(ring.head + ring.n) % 4] = slot;
  ring.bound[(ring.head + ring.n) % 4] = l + 1;
  ++ring.n;
  while (ring.n > 2) {
    const int sl = ring.slot[ring.head];
    e = hipEventSynchronize(net->events[(size_t)sl]);
    if (e != hipSuccess) return e;
    ring.head = (ring.head + 1) % 4;
    --ring.n;
    *live_bound = std::min<int64_t>(*live_bound, net->pinned[sl]);
  }
  return hipSuccess;
}

// Report of a compaction enqueued with a tag (see k_compact): the live count and the flags.
struct Report {
  int64_t count = 0;
  bool nonbinary = false, overflow = false;
};

// Tag for the next reporting compaction (24 bits, never 0: the word starts at 0).
unsigned long long next_report_tag(sdnn_net *net) {
  net->notify_seq = (net->notify_seq + 1) & 0xffffffu;
  if (net->notify_seq == 0) net->notify_seq = 1;
  return net->notify_seq;
}

// Wait for the report tagged `tag`: spin on the word in coherent host memory (no OS wake-up in the
// way); if none arrives within 2 s, wait for the stream and read the count (at count_dev) and the
// flags by copies.
hipError_t wait_report(sdnn_net *net, unsigned long long tag, const int *count_dev, Report *r) {
  const auto t0 = std::chrono::steady_clock::now();
  for (uint32_t it = 1;; ++it) {
    const unsigned long long w = __atomic_load_n(net->notify, __ATOMIC_ACQUIRE);
    if ((w >> 40) == tag) {
      r->count = (int64_t)(w & 0xffffffffull);
      r->nonbinary = ((w >> 32) & 1ull) != 0;
      r->overflow = ((w >> 33) & 1ull) != 0;
      return hipSuccess;
    }
    if ((it & 4095u) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(2)) break;
    __builtin_ia32_pause();
  }
  hipError_t e = hipStreamSynchronize(net->stream);
  if (e != hipSuccess) return e;
  int32_t v[3] = {0, 0, 0};
  e = hipMemcpy(&v[0], count_dev, sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(&v[1], net->misc, sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(&v[2], net->misc + kOverflowSlot, sizeof(int32_t), hipMemcpyDeviceToHost);
  r->count = v[0];
  r->nonbinary = v[1] != 0;
  r->overflow = v[2] != 0;
  return e;
}

// LDS-tile path: row-major activations ping-pong between two buffers; the live list is compacted
// after every layer.
sdnn_status infer_lds(sdnn_net *net, const float *y0, int M) {
  hipStream_t s = net->stream;
  const float *yin = y0;
  int cur = 0;
  int32_t l = 0;
  int64_t live_bound = M;
  // One launch runs every remaining layer once the live rows fit one workgroup per CU and either
  // take 4-row tiles or have stopped dying fast (the last two layers, not counting layer 0, each
  // kept 90% of their rows): inside that launch dead rows still occupy their tile's slots, while
  // layer-by-layer launches compact them away. Until the switch the count is read back after each
  // layer (those layers are long).
  const int bmax = fused_rows_max(net);
  int kept = 0;  // consecutive layers after layer 0 that kept at least 90% of their rows
  for (; l < net->L && live_bound > 0; ++l) {
    float *yout = net->ybuf[l & 1];
    const bool fits = (live_bound + bmax - 1) / bmax <= net->cus;
    const bool settled = kept >= 2;
    if (l > 0 && (live_bound <= 4 * (int64_t)net->cus || (fits && settled))) {
      const bool rec = net->profiling;
      if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_start[(size_t)l], s));
      HIP_OR_POISON(net, launch_layers_lds(net, yin, yout, l, net->ids[cur], net->counts + l, live_bound));
      if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_end[(size_t)l], s));
      if (net->profiling) net->prof_rec[(size_t)l] = rec;
      for (int32_t q = l; q < net->L; ++q) {
        net->layer_kernel[(size_t)q] = SDNN_KERNEL_LDS_FUSED;
        net->layer_launches[(size_t)q] = q == l ? 1 : 0;
      }
      // the final list: positions still live after the last layer (bits per 32 positions)
      hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, net->masks, 32, net->ids[cur], net->ids[cur ^ 1],
                         (int *)nullptr, net->counts + l, net->counts + net->L, (int *)nullptr, (const int *)nullptr,
                         (unsigned long long *)nullptr, 0ull);
      HIP_OR_POISON(net, hipGetLastError());
      cur ^= 1;
      net->layers_run = net->L;
      net->final_list = cur;
      net->final_y = yout;
      net->final_fm = nullptr;
      return SDNN_OK;
    }
    const bool rec = net->profiling && (net->prof_mode == 1 || live_bound > 256);
    if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_start[(size_t)l], s));
    // layer 0 of a uniform layer on a large batch (from 2^24 inputs, where packing and a read-back
    // cost less than they save): if every input is 0 or 1, by counts of the bit-packed rows (see
    // k_layer_count), written back as fp32 rows; masks then hold one bit per list position
    int mask_rows = net->B;
    bool counted = false;
    const LayerDev &ld0 = net->layers[0];
    if (l == 0 && (int64_t)M * net->N >= (1 << 24) && ld0.uniform && ld0.ell16 && ld0.w > 0.0f && (net->N & 3) == 0 &&
        (uint64_t)M * (uint64_t)net->N / 4 < (1ull << 32)) {
      HIP_OR_POISON(net, launch_pack_bits<32>(net, y0, net->ybuf[1], net->ids[cur], net->counts));
      HIP_OR_POISON(net, hipMemcpyAsync(net->pinned + 6, net->misc, sizeof(int32_t), hipMemcpyDeviceToHost, s));
      HIP_OR_POISON(net, hipStreamSynchronize(s));
      if (net->pinned[6] == 0) {
        HIP_OR_POISON(net, (launch_layer_count_k<32, true>(net, ld0, net->ybuf[1], nullptr, net->counts, yout,
                                                           net->ids[cur], net->masks)));
        counted = true;
        mask_rows = 32;
      }
    }
    if (!counted)
      HIP_OR_POISON(net, launch_layer(net, l, yin, yout, net->ids[cur], net->counts + l, l == 0 ? net->rownz : nullptr));
    if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_end[(size_t)l], s));
    net->layer_kernel[(size_t)l] = counted ? SDNN_KERNEL_BITS_COUNT : SDNN_KERNEL_LDS_TILE;
    net->layer_launches[(size_t)l] = counted ? 3 : 1;
    if (net->profiling) net->prof_rec[(size_t)l] = rec;
    const unsigned long long tag = next_report_tag(net);
    hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, net->masks, mask_rows, net->ids[cur], net->ids[cur ^ 1],
                       (int *)nullptr, net->counts + l, net->counts + l + 1, (int *)nullptr, net->misc,
                       net->notify_dev, tag);
    HIP_OR_POISON(net, hipGetLastError());
    cur ^= 1;
    yin = yout;
    Report rp;
    HIP_OR_POISON(net, wait_report(net, tag, net->counts + l + 1, &rp));
    const int64_t before = live_bound;
    live_bound = std::min<int64_t>(live_bound, rp.count);
    kept = (l > 0 && live_bound * 10 >= before * 9) ? kept + 1 : 0;
  }
  net->layers_run = l;
  net->final_list = cur;
  net->final_y = (l == net->L && net->L > 0) ? net->ybuf[(net->L - 1) & 1] : nullptr;
  net->final_fm = nullptr;
  return SDNN_OK;
}

// Global-tile path: activations stay in feature-major tiles of 32 list positions from layer to
// layer. Large layers are followed by a compaction of the live list (ids plus each live row's old
// position); the tiles are repacked to the compacted list only when that saves tiles, otherwise the
// next layer runs on the old positions, where rows that died hold zeros and stay zero. Small layers
// (one round of tiles) count their live rows themselves, so a layer is one launch; they are
// compacted only when the live bound says that fewer tiles would do, and after the last layer.
// Liveness masks alternate between two buffers by layer parity.
sdnn_status infer_gfm(sdnn_net *net, const float *y0, int M) {
  hipStream_t s = net->stream;
  int *npos = net->misc + kNposSlot;  // npos[i]: positions in list i
  const int64_t one_round = 8 * 32;
  auto tiles = [](int64_t r) { return (r + 31) / 32; };
  auto masks_for = [net](int32_t layer) { return net->masks_rot[layer % 3]; };
  int cur = 0;
  int64_t P = M;           // host bound on the positions of list cur (exact after a read-back)
  int64_t live_bound = M;  // host bound on the live rows
  const float *fin = nullptr;
  float *fout = nullptr;
  bool fin_codes = false, fout_codes = false;  // the tiles hold dictionary codes
  bool fin_wide = false;  // fin's codes are two bytes (k_encode<64, 2>), else one
  bool wide_ok = true;    // a two-byte encoding is worth trying
  bool next_tried = false;     // the repack after this layer tried one-byte codes for the next layer
  bool repacked_codes = false;  // ... and wrote them (else fp32 tiles)
  int last_list = 0;
  bool compacted = true;   // the last layer run has been followed by a compaction
  PollRing ring;
  // few-tile layers leave their liveness in partial words; the next few-tile launch turns them into
  // mask words, any other reader of the masks needs k_finalize_masks first
  bool parts_pending = false;
  int32_t part_layer = -1;
  int part_S = 0, part_nt = 0;
  auto finalize_parts = [&]() -> hipError_t {
    if (!parts_pending) return hipSuccess;
    parts_pending = false;
    hipLaunchKernelGGL(k_finalize_masks, dim3(1), dim3(kPartThreads), 0, s, net->part[part_layer & 1], part_S, part_nt,
                       masks_for(part_layer));
    return hipGetLastError();
  };
  // few-tile layers: the host follows the device through the progress word, staying at most
  // kProgressAhead layers ahead of it, so that it learns within a few layers that no row is left
  const unsigned long long gen = net->run_gen & 0xffffu;
  bool follow = net->progress != nullptr;
  auto follow_progress = [&](int32_t layer) -> hipError_t {
    const int32_t need = layer - kProgressAhead;
    if (!follow || need < 0) return hipSuccess;
    const auto t0 = std::chrono::steady_clock::now();
    for (uint32_t it = 1;; ++it) {
      const unsigned long long w = __atomic_load_n(net->progress, __ATOMIC_ACQUIRE);
      if ((w >> kProgGenShift) == gen && (int32_t)((w >> kProgLayerShift) & 0xfffffu) >= need) {
        const unsigned long long c = w & kProgCountMask;
        if (c != kProgCountMask) live_bound = std::min<int64_t>(live_bound, (int64_t)c);
        return hipSuccess;
      }
      if ((it & 4095u) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::seconds(2)) {
        // no report from the device: wait for the stream, and poll by copies from now on
        follow = false;
        return hipStreamSynchronize(s);
      }
      __builtin_ia32_pause();
    }
  };
  bool bits_route = false;  // layer 0 went to the bit-tile kernels (unless the report says otherwise)
  int32_t l = 0;
  for (; l < net->L && live_bound > 0; ++l) {
    const bool small = l > 0 && P <= one_round;
    bool reported = false;  // this layer's launch writes the progress word
    fout_codes = false;
    // the columns fout holds, when this layer computed one column per group of equal columns
    const LayerDev &lcur = net->layers[(size_t)l];
    const bool ocols_on = lcur.K == 32 && lcur.src16 && lcur.cols && lcur.dedup_ok;
    const int *fout_cols = nullptr;  // set by the branches whose kernels take the column list
    bool spread_used = false;  // this layer's liveness is in the spread words
    bool seglive_out = false;  // fout's all-zero segments were skipped (net->seglive says which)
    unsigned *mk = masks_for(l);
    const bool rec = net->profiling && (net->prof_mode == 1 || !small);
    if (net->profiling) net->prof_rec[(size_t)l] = rec;
    if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_start[(size_t)l], s));
    bool encoded = false;  // this layer reads codes that k_encode wrote from fp32 tiles
    int encode_tries = 0;  // launches spent on encodings of this layer's inputs
    const bool tried = next_tried;  // the repack before this layer tried one-byte codes (they overflowed)
    next_tried = false;
    repacked_codes = false;
    if (l > 0 && !fin_codes && compacted && live_bound >= kEncodeMinRows && !net->equal_value_kernels) {
      // a large layer on fp32 tiles: if its inputs take at most 256 distinct values (saturated rows
      // do), encode them as one-byte codes into the free buffer and gather those instead (unless the
      // repack before this layer found that they do not fit: tried); else, if
      // they take at most 4096 and the fp32 tiles outgrow the L2 (kXcdL2Bytes), as two-byte codes;
      // a full dictionary stops an encoding early, and when both stop the layer reads the fp32 tiles
      unsigned char *cbuf = reinterpret_cast<unsigned char *>((fin == net->fm[1]) ? net->fm[0] : net->fm[1]);
      auto try_encode = [&](int cb) -> hipError_t {
        unsigned *gd = cb == 1 ? net->dict : net->dict16;
        if (cb == 1)
          hipLaunchKernelGGL(k_dict_reset<1>, dim3(1), dim3(256), 0, s, gd, net->misc + kOverflowSlot);
        else
          hipLaunchKernelGGL(k_dict_reset<2>, dim3(16), dim3(256), 0, s, gd, net->misc + kOverflowSlot);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int cr = code_rows(net->bitsT);
        const int64_t items = (live_bound + cr - 1) / cr * (int64_t)net->N * (cr / 16);
        const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus * 8, (items + 255) / 256));
        if (cb == 2 && cr != 64) return hipErrorInvalidValue;
        if (cb == 2)
          hipLaunchKernelGGL((k_encode<64, 2>), dim3(grid), dim3(256), 0, s, fin, cbuf, net->N, npos + cur, gd,
                             net->misc + kOverflowSlot);
        else if (cr == 128)
          hipLaunchKernelGGL((k_encode<128, 1>), dim3(grid), dim3(256), 0, s, fin, cbuf, net->N, npos + cur, gd,
                             net->misc + kOverflowSlot);
        else
          hipLaunchKernelGGL((k_encode<64, 1>), dim3(grid), dim3(256), 0, s, fin, cbuf, net->N, npos + cur, gd,
                             net->misc + kOverflowSlot);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const unsigned long long tag = next_report_tag(net);
        hipLaunchKernelGGL(k_report_overflow, dim3(1), dim3(1), 0, s, net->misc + kOverflowSlot, net->notify_dev, tag);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        Report rp;
        e = wait_report(net, tag, npos + cur, &rp);
        if (e != hipSuccess) return e;
        encode_tries += 3;
        if (!rp.overflow) {
          fin = reinterpret_cast<const float *>(cbuf);
          fin_codes = true;
          fin_wide = cb == 2;
          encoded = true;
          if (cb == 1) wide_ok = true;
        }
        return hipSuccess;
      };
      if (!tried) HIP_OR_POISON(net, try_encode(1));
      if (!encoded && net->dict16 && wide_ok && (size_t)net->N * 32 * sizeof(float) > kXcdL2Bytes) {
        HIP_OR_POISON(net, try_encode(2));
        // inputs with more than 4096 values: the layers after it are not tried again until the
        // inputs of one of them fit 256 values (values that grow more varied stay so for a while)
        if (!encoded) wide_ok = false;
      }
    }
    fout = (fin == net->fm[1]) ? net->fm[0] : net->fm[1];
    if (l == 0) {
      // layer 0 reads the caller's rows; binary inputs go through bit tiles (built in fm[0]),
      // others through feature-major tiles in fm[0]; both passes also find the nonzero input rows
      // the pack pass addresses rows with 32-bit offsets (in floats, or float4 when N % 4 == 0)
      const uint64_t units = (uint64_t)M * (uint64_t)net->N / ((net->N & 3) == 0 ? 4 : 1);
      const bool try_bits = net->bitsT > 0 && net->layers[0].K <= 32 && net->layers[0].ellw && units < (1ull << 32) &&
                            (net->bitsT == 32 ? bits_tile_bytes_needed<32>(net) <= bits_tile_bytes(32)
                                              : bits_tile_bytes_needed<16>(net) <= bits_tile_bytes(16));
      if (try_bits) {
        // the bit-tile kernels that follow exit at once if the pack finds an input other than 0 or 1
        // (misc[0]); the host learns of it from the layer's compaction report and then computes
        // layer 0 on fp32 tiles (no host round trip inside the layer)
        HIP_OR_POISON(net, net->bitsT == 32 ? launch_pack_bits<32>(net, y0, net->fm[0], net->ids[cur], npos + cur)
                                            : launch_pack_bits<16>(net, y0, net->fm[0], net->ids[cur], npos + cur));
        bits_route = true;
      }
      const LayerDev &ld0 = net->layers[0];
      if (bits_route && P > one_round && net->L > 1 && ld0.uniform && ld0.ell16 && ld0.w > 0.0f) {
        // a uniform layer: the output of a column is a function of how many of its sources are 1,
        // so the counts are the codes (see k_layer_count)
        fout_codes = true;
        net->layer_kernel[0] = SDNN_KERNEL_BITS_COUNT;
        net->layer_launches[0] = 3;  // pack + dictionary + count
        unsigned char *cout = reinterpret_cast<unsigned char *>(fout);
        HIP_OR_POISON(net, net->bitsT == 32 ? launch_layer_count<32>(net, ld0, net->fm[0], cout, npos + cur)
                                            : launch_layer_count<16>(net, ld0, net->fm[0], cout, npos + cur));
      } else if (bits_route) {
        // outputs of a layer on binary inputs take few distinct values: a large layer 0 writes them
        // as one-byte dictionary codes, which the next layer gathers four times denser
        fout_codes = P > one_round && net->L > 1;
        net->layer_kernel[0] = fout_codes ? SDNN_KERNEL_BITS_TO_CODES : SDNN_KERNEL_BITS;
        net->layer_launches[0] = 2;  // pack + layer
        HIP_OR_POISON(net, net->bitsT == 32
                               ? launch_layer_bits<32>(net, net->layers[0], net->fm[0], fout, npos + cur, fout_codes)
                               : launch_layer_bits<16>(net, net->layers[0], net->fm[0], fout, npos + cur, fout_codes));
      } else {
        HIP_OR_POISON(net, launch_to_fm(net, y0, net->fm[0], net->ids[cur], npos + cur, try_bits ? nullptr : net->rownz));
        HIP_OR_POISON(net, launch_gfm(net, net->layers[0], net->fm[0], fout, npos + cur, tiles(P), mk, nullptr, nullptr,
                                      nullptr, net->spread));
        spread_used = true;
        fout_cols = ocols_on ? lcur.cols : nullptr;
        net->layer_kernel[0] = SDNN_KERNEL_GLOBAL_TILE;
        net->layer_launches[0] = 1 + gfm_launches(net, net->layers[0], tiles(P), 0) + (try_bits ? 1 : 0);
      }
    } else if (fin_codes) {
      // follows layer 0 or a layer whose outputs were encoded, both compacted: no count to take over
      const unsigned char *cin = reinterpret_cast<const unsigned char *>(fin);
      if (fin_wide)
        HIP_OR_POISON(net, launch_gfm_u16(net, net->layers[(size_t)l], cin, fout, npos + cur, tiles(P), mk, &seglive_out));
      else
        HIP_OR_POISON(net, launch_gfm_u8(net, net->layers[(size_t)l], cin, fout, npos + cur, tiles(P), mk, &seglive_out));
      spread_used = true;
      fout_cols = ocols_on ? lcur.cols : nullptr;
      net->layer_kernel[(size_t)l] = fin_wide ? SDNN_KERNEL_GLOBAL_TILE_CODES16 : SDNN_KERNEL_GLOBAL_TILE_CODES;
      const int st = code_rows(net->bitsT) / 32;  // fp32 tiles per code tile
      // (with the dictionary resets, encodings and their reports when this layer encoded its inputs)
      net->layer_launches[(size_t)l] = gfm_launches(net, net->layers[(size_t)l], tiles(P), st * 32) + encode_tries;
    } else {
      // after a layer without compaction, this launch counts that layer's live rows
      const LayerDev &ld = net->layers[(size_t)l];
      int *cnt = compacted ? nullptr : net->counts + l;
      if (small && ld.K == 32) {
        const unsigned *prev = cnt && parts_pending ? net->part[part_layer & 1] : nullptr;
        int S = 0, nt = 0;
        const unsigned long long tag = (gen << kProgGenShift) | ((unsigned long long)l << kProgLayerShift);
        HIP_OR_POISON(net, launch_gfm_small(net, ld, fin, fout, npos + cur, tiles(P), net->part[l & 1], prev, part_S,
                                            part_nt, masks_for(l - 1), masks_for(l + 1), cnt, net->counts + (l - 1),
                                            follow ? net->progress_dev : nullptr, tag, &S, &nt));
        reported = follow;
        fout_cols = ocols_on ? lcur.cols : nullptr;
        parts_pending = true;
        part_layer = l;
        part_S = S;
        part_nt = nt;
        net->layer_kernel[(size_t)l] = SDNN_KERNEL_GLOBAL_TILE_FEW_ROWS;
        net->layer_launches[(size_t)l] = 1;
      } else {
        HIP_OR_POISON(net, finalize_parts());
        // a large layer's liveness goes through spread words (compacted right after)
        HIP_OR_POISON(net, launch_gfm(net, ld, fin, fout, npos + cur, tiles(P), mk, masks_for(l - 1),
                                      masks_for(l + 1), cnt, small ? nullptr : net->spread));
        spread_used = !small;
        fout_cols = ocols_on ? lcur.cols : nullptr;
        net->layer_kernel[(size_t)l] = SDNN_KERNEL_GLOBAL_TILE;
        net->layer_launches[(size_t)l] = gfm_launches(net, ld, tiles(P), 0) + encode_tries;
      }
    }
    if (rec) HIP_OR_POISON(net, hipEventRecord(net->prof_end[(size_t)l], s));
    // compaction of this layer's live rows; with tag != 0 it reports its count and flags
    auto compact = [&](unsigned long long tag = 0) -> hipError_t {
      hipError_t e = finalize_parts();
      if (e != hipSuccess) return e;
      if (spread_used) {
        const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus, (tiles(P) + 255) / 256));
        hipLaunchKernelGGL(k_spread_to_masks, dim3(grid), dim3(256), 0, s, net->spread, npos + cur, mk);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        spread_used = false;
      }
      hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, mk, 32, net->ids[cur], net->ids[cur ^ 1],
                         net->src[cur ^ 1], npos + cur, net->counts + l + 1, npos + (cur ^ 1), net->misc,
                         tag ? net->notify_dev : nullptr, tag);
      last_list = cur ^ 1;
      return hipGetLastError();
    };
    // the repack of this layer's outputs as the next layer's one-byte codes (k_repack<1, CR>), into
    // dst; sets repacked_codes when the dictionary held every value
    auto repack_codes = [&](float *dst) -> hipError_t {
      unsigned *gd = net->dict;
      hipLaunchKernelGGL(k_dict_reset<1>, dim3(1), dim3(256), 0, s, gd, net->misc + kOverflowSlot);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      const int cr = code_rows(net->bitsT);
      const int64_t items = (live_bound + cr - 1) / cr * (cr / 32) * ((net->N + kRepackSources - 1) / kRepackSources);
      const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus * 8, items));
      unsigned char *dc = reinterpret_cast<unsigned char *>(dst);
      const unsigned *sl = seglive_out ? net->seglive : nullptr;
      int *of = net->misc + kOverflowSlot;
      const int *sp = net->src[cur ^ 1], *np = npos + (cur ^ 1);
      if (cr == 128)
        hipLaunchKernelGGL((k_repack<1, 128>), dim3(grid), dim3(256), 0, s, fout, (float *)nullptr, net->N, sp, np, sl,
                           (const int *)nullptr, net->N, dc, gd, of);
      else
        hipLaunchKernelGGL((k_repack<1, 64>), dim3(grid), dim3(256), 0, s, fout, (float *)nullptr, net->N, sp, np, sl,
                           (const int *)nullptr, net->N, dc, gd, of);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      const unsigned long long tag = next_report_tag(net);
      hipLaunchKernelGGL(k_report_overflow, dim3(1), dim3(1), 0, s, of, net->notify_dev, tag);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      Report rp;
      e = wait_report(net, tag, np, &rp);
      if (e == hipSuccess && !rp.overflow) repacked_codes = true;
      return e;
    };
    compacted = false;
    bool adopt;
    if (!small) {
      // a large layer: compact, and wait for its exact count (the next layer is large, so the wait
      // is short relative to it)
      unsigned long long tag = next_report_tag(net);
      HIP_OR_POISON(net, compact(tag));
      compacted = true;
      Report rp;
      HIP_OR_POISON(net, wait_report(net, tag, net->counts + l + 1, &rp));
      if (l == 0 && bits_route && rp.nonbinary) {
        // an input is not 0 or 1: the bit-tile kernel exited at once; layer 0 on fp32 tiles
        fout_codes = false;
        HIP_OR_POISON(net, launch_to_fm(net, y0, net->fm[0], net->ids[cur], npos + cur, nullptr));
        HIP_OR_POISON(net, launch_gfm(net, net->layers[0], net->fm[0], fout, npos + cur, tiles(P), mk, nullptr,
                                      nullptr, nullptr, net->spread));
        spread_used = true;
        net->layer_kernel[0] = SDNN_KERNEL_GLOBAL_TILE;
        net->layer_launches[0] = 2 + gfm_launches(net, net->layers[0], tiles(P), 0);
        tag = next_report_tag(net);
        HIP_OR_POISON(net, compact(tag));
        HIP_OR_POISON(net, wait_report(net, tag, net->counts + l + 1, &rp));
      } else if (fout_codes && rp.overflow) {
        // more than 256 distinct values: redo layer 0 with fp32 outputs (same liveness)
        fout_codes = false;
        net->layer_kernel[0] = SDNN_KERNEL_BITS;
        net->layer_launches[0] = 3;  // pack + the layer with codes + the layer again with fp32 outputs
        HIP_OR_POISON(net, net->bitsT == 32
                               ? launch_layer_bits<32>(net, net->layers[0], net->fm[0], fout, npos + cur, false)
                               : launch_layer_bits<16>(net, net->layers[0], net->fm[0], fout, npos + cur, false));
        tag = next_report_tag(net);
        HIP_OR_POISON(net, compact(tag));
        HIP_OR_POISON(net, wait_report(net, tag, net->counts + l + 1, &rp));
      }
      live_bound = std::min<int64_t>(live_bound, rp.count);
      adopt = live_bound == 0 || tiles(live_bound) * 20 <= tiles(P) * 19;
    } else {
      adopt = tiles(live_bound) < tiles(P);
    }
    if (adopt && live_bound > 0 && l + 1 < net->L) {
      if (!compacted) HIP_OR_POISON(net, compact());
      compacted = true;
      float *dst = (fout == net->fm[1]) ? net->fm[0] : net->fm[1];
      const int cr = code_rows(net->bitsT);
      const int64_t items = fout_codes ? (tiles(live_bound) + cr / 32 - 1) / (cr / 32) * net->N * (cr / 4) / 256
                                       : tiles(live_bound) * (((fout_cols ? lcur.D : net->N) + kRepackSources - 1) /
                                                              kRepackSources);
      const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus * 8, items));
      if (fout_codes && cr == 128)
        hipLaunchKernelGGL(k_repack_u8<128>, dim3(grid), dim3(256), 0, s, reinterpret_cast<const unsigned char *>(fout),
                           reinterpret_cast<unsigned char *>(dst), net->N, net->src[cur ^ 1], npos + (cur ^ 1));
      else if (fout_codes)
        hipLaunchKernelGGL(k_repack_u8<64>, dim3(grid), dim3(256), 0, s, reinterpret_cast<const unsigned char *>(fout),
                           reinterpret_cast<unsigned char *>(dst), net->N, net->src[cur ^ 1], npos + (cur ^ 1));
      else {
        // the next layer encodes its inputs if they fit a dictionary (see the start of the loop):
        // the repack writes one-byte codes itself, and falls back to fp32 tiles when they overflow
        // (two-byte codes are then tried by k_encode from the fp32 tiles: written by the repack
        // they measured slower, 30.9 ms per step against 30.4 at 65536 neurons and 60,000 inputs)
        if (live_bound >= kEncodeMinRows && !net->equal_value_kernels && !fout_cols) {
          next_tried = true;
          HIP_OR_POISON(net, repack_codes(dst));
          if (repacked_codes) wide_ok = true;
        }
        if (!repacked_codes)
          hipLaunchKernelGGL((k_repack<0, 32>), dim3(grid), dim3(256), 0, s, fout, dst, net->N, net->src[cur ^ 1],
                             npos + (cur ^ 1), seglive_out ? net->seglive : nullptr, fout_cols,
                             fout_cols ? lcur.D : net->N, (unsigned char *)nullptr, (unsigned *)nullptr, (int *)nullptr);
      }
      HIP_OR_POISON(net, hipGetLastError());
      fin = dst;
      cur ^= 1;
      P = live_bound;
    } else {
      if (seglive_out) {
        // the next layer (or the final read-out) takes the tiles as they are
        const int64_t items = tiles(P) * net->N * 8;
        const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus * 8, (items + 255) / 256));
        hipLaunchKernelGGL(k_fill_dead, dim3(grid), dim3(256), 0, s, fout, net->N, net->seglive, npos + cur);
        HIP_OR_POISON(net, hipGetLastError());
      }
      fin = fout;
    }
    fin_codes = fout_codes || repacked_codes;  // (one-byte codes: a layer or a repack writes no others)
    fin_wide = false;
    // counts[l] is final once layer l has run (written by a compaction or by layer l's launch)
    if (reported)
      HIP_OR_POISON(net, follow_progress(l));
    else
      HIP_OR_POISON(net, poll_step(net, ring, l, l, &live_bound));
  }
  if (!compacted) {
    // the final list: compaction of the last layer's masks
    const int32_t last = l - 1;
    HIP_OR_POISON(net, finalize_parts());
    hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, masks_for(last), 32, net->ids[cur], net->ids[cur ^ 1],
                       net->src[cur ^ 1], npos + cur, net->counts + last + 1, npos + (cur ^ 1), (const int *)nullptr,
                       (unsigned long long *)nullptr, 0ull);
    HIP_OR_POISON(net, hipGetLastError());
    last_list = cur ^ 1;
  }
  net->layers_run = l;
  net->final_list = last_list;
  net->final_y = nullptr;
  net->final_fm = (l == net->L && net->L > 0) ? fout : nullptr;
  return SDNN_OK;
}

sdnn_status infer_impl(sdnn_net *net, const float *y0, int64_t n_rows, void *workspace, size_t workspace_bytes,
                       void *hip_stream);

}  // namespace

sdnn_status sdnn_infer(sdnn_net *net, const float *y0, int64_t n_rows, void *workspace, size_t workspace_bytes,
                       void *hip_stream) {
  return infer_impl(net, y0, n_rows, workspace, workspace_bytes, hip_stream);
}

sdnn_status sdnn_infer_static(sdnn_net *net, const float *y0, int64_t n_rows, void *hip_stream) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (n_rows < 0) return fail(SDNN_EINVAL, "n_rows %lld out of range", (long long)n_rows);
  const size_t need = sdnn_workspace_bytes(net, n_rows);
  if (need > kStaticWorkspaceBytes)
    return fail(SDNN_ERANGE, "%lld rows need %zu bytes of workspace; the static workspace holds %zu",
                (long long)n_rows, need, kStaticWorkspaceBytes);
  int dev = -1;
  HIP_OR_POISON(net, hipGetDevice(&dev));
  void *ws = nullptr;
  st = scratch_address(dev, &ws);
  if (st != SDNN_OK) return st;
  return infer_impl(net, y0, n_rows, ws, kStaticWorkspaceBytes, hip_stream);
}


namespace {

sdnn_status infer_impl(sdnn_net *net, const float *y0, int64_t n_rows, void *workspace, size_t workspace_bytes,
                       void *hip_stream) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (net->n_loaded != net->L) return fail(SDNN_ESTATE, "%d of %d layers loaded", net->n_loaded, net->L);
  if (n_rows < 0 || n_rows > (int64_t)0x7fffffff) return fail(SDNN_EINVAL, "n_rows %lld out of range", (long long)n_rows);
  if (n_rows > 0 && !y0) return fail(SDNN_EINVAL, "y0 is null");
  if (!workspace) return fail(SDNN_EINVAL, "workspace is null");
  if (reinterpret_cast<uintptr_t>(workspace) % 256) return fail(SDNN_EINVAL, "workspace is not 256-byte aligned");
  if (n_rows > 0 && reinterpret_cast<uintptr_t>(y0) % 16 && net->N % 4 == 0)
    return fail(SDNN_EINVAL, "y0 must be 16-byte aligned");
  const WsLayout w = layout_for(net, n_rows);
  if (workspace_bytes < w.total) return fail(SDNN_EINVAL, "workspace has %zu bytes, needs %zu", workspace_bytes, w.total);
  int dev = -1;
  HIP_OR_POISON(net, hipGetDevice(&dev));
  if (dev != net->device) return fail(SDNN_EINVAL, "current device %d differs from the handle's device %d", dev, net->device);
  char *ws = static_cast<char *>(workspace);
  net->M = n_rows;
  ++net->run_gen;
  net->stream = reinterpret_cast<hipStream_t>(hip_stream);
  net->ws = ws;
  for (int i = 0; i < 2; ++i) {
    float *act = reinterpret_cast<float *>(ws + w.act[i]);
    net->ybuf[i] = net->path == 0 ? act : nullptr;
    net->fm[i] = net->path == 1 ? act : nullptr;
    net->ids[i] = reinterpret_cast<int *>(ws + w.ids[i]);
    net->src[i] = reinterpret_cast<int *>(ws + w.src[i]);
  }
  for (int i = 0; i < 3; ++i) net->masks_rot[i] = reinterpret_cast<unsigned *>(ws + w.masks[i]);
  net->masks = net->masks_rot[0];
  net->rownz = reinterpret_cast<int *>(ws + w.rownz);
  net->counts = reinterpret_cast<int *>(ws + w.counts);
  net->misc = reinterpret_cast<int *>(ws + w.misc);
  net->dict = reinterpret_cast<unsigned *>(ws + w.dict);
  net->dict16 = net->path == 1 ? reinterpret_cast<unsigned *>(ws + w.dict16) : nullptr;
  net->seglive = reinterpret_cast<unsigned *>(ws + w.seglive);
  for (int i = 0; i < 2; ++i) net->part[i] = reinterpret_cast<unsigned *>(ws + w.part[i]);
  net->spread = reinterpret_cast<unsigned *>(ws + w.spread);
  net->final_ids = reinterpret_cast<long long *>(ws + w.final_ids);
  net->ran = false;

  const int M = (int)n_rows;
  hipStream_t s = net->stream;
  hipLaunchKernelGGL(k_init, dim3(std::max(1, std::min(net->cus * 4, (M + 255) / 256 + 1))), dim3(256), 0, s,
                     net->ids[0], net->masks_rot[0], net->masks_rot[1], net->masks_rot[2], net->rownz, net->counts,
                     net->misc, net->dict, M, net->L, net->spread, w.spread_words);
  HIP_OR_POISON(net, hipGetLastError());
  if (net->profiling) net->prof_rec.assign((size_t)net->L, 0);
  net->layer_kernel.assign((size_t)net->L, SDNN_KERNEL_NONE);
  net->layer_launches.assign((size_t)net->L, 0);
  st = net->path == 0 ? infer_lds(net, y0, M) : infer_gfm(net, y0, M);
  if (st != SDNN_OK) return st;
  hipLaunchKernelGGL(k_final_ids, dim3(std::max(1, std::min(net->cus, (M + 255) / 256 + 1))), dim3(256), 0, s,
                     net->ids[net->final_list], net->counts + net->layers_run, net->final_ids);
  HIP_OR_POISON(net, hipGetLastError());
  net->ran = true;
  net->pending_times = net->profiling;
  g_err.clear();
  return SDNN_OK;
}

}  // namespace

sdnn_status sdnn_categories(sdnn_net *net, int64_t *ids, int64_t capacity, int64_t *count) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (!net->ran) return fail(SDNN_ESTATE, "no inference has run");
  if (!count) return fail(SDNN_EINVAL, "count is null");
  HIP_OR_POISON(net, hipStreamSynchronize(net->stream));
  if (net->pending_times) {
    for (int32_t l = 0; l < net->layers_run; ++l) {
      if (!net->prof_rec[(size_t)l]) continue;
      float ms = 0.0f;
      HIP_OR_POISON(net, hipEventElapsedTime(&ms, net->prof_start[(size_t)l], net->prof_end[(size_t)l]));
      net->prof_ms[(size_t)l] += ms;
      net->prof_runs[(size_t)l] += 1;
    }
    net->pending_times = false;
  }
  int32_t c = 0;
  HIP_OR_POISON(net, hipMemcpy(&c, net->counts + net->layers_run, sizeof(int32_t), hipMemcpyDeviceToHost));
  *count = c;
  if (!ids || capacity < c) return fail(SDNN_ERANGE, "need capacity %d", c);
  if (c > 0) HIP_OR_POISON(net, hipMemcpy(ids, net->final_ids, (size_t)c * sizeof(long long), hipMemcpyDeviceToHost));
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_live_counts(sdnn_net *net, int64_t *counts) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (!net->ran) return fail(SDNN_ESTATE, "no inference has run");
  if (!counts) return fail(SDNN_EINVAL, "counts is null");
  HIP_OR_POISON(net, hipStreamSynchronize(net->stream));
  std::vector<int32_t> c((size_t)net->L + 1);
  HIP_OR_POISON(net, hipMemcpy(c.data(), net->counts, c.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  std::vector<int32_t> nz((size_t)std::max<int64_t>(net->M, 1));
  if (net->M > 0) HIP_OR_POISON(net, hipMemcpy(nz.data(), net->rownz, (size_t)net->M * sizeof(int32_t), hipMemcpyDeviceToHost));
  int64_t r0 = 0;
  for (int64_t i = 0; i < net->M; ++i) r0 += nz[(size_t)i] != 0;
  counts[0] = r0;
  for (int32_t l = 1; l <= net->L; ++l) counts[l] = c[(size_t)l];
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_final_rows(sdnn_net *net, const int64_t *ids, int64_t n, float *out_host) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (!net->ran) return fail(SDNN_ESTATE, "no inference has run");
  if (n < 0 || (n > 0 && (!ids || !out_host))) return fail(SDNN_EINVAL, "bad arguments");
  for (int64_t q = 0; q < n; ++q)
    if (ids[q] < 0 || ids[q] >= net->M) return fail(SDNN_EINVAL, "row id %lld out of range", (long long)ids[q]);
  HIP_OR_POISON(net, hipStreamSynchronize(net->stream));
  int32_t c = 0;
  HIP_OR_POISON(net, hipMemcpy(&c, net->counts + net->layers_run, sizeof(int32_t), hipMemcpyDeviceToHost));
  std::vector<long long> live((size_t)std::max(c, 1));
  if (c > 0) HIP_OR_POISON(net, hipMemcpy(live.data(), net->final_ids, (size_t)c * sizeof(long long), hipMemcpyDeviceToHost));
  const size_t rowb = (size_t)net->N * sizeof(float);
  if (net->path == 0) {
    for (int64_t q = 0; q < n; ++q) {
      float *dst = out_host + (size_t)q * net->N;
      const bool is_live = c > 0 && net->final_y && std::binary_search(live.begin(), live.begin() + c, (long long)ids[q]);
      if (is_live) {
        HIP_OR_POISON(net, hipMemcpy(dst, net->final_y + (size_t)ids[q] * net->N, rowb, hipMemcpyDeviceToHost));
        // the last layer may have computed only one column of each group of equal columns
        if (!net->last_rep.empty())
          for (int32_t j = 0; j < net->N; ++j) dst[j] = dst[net->last_rep[(size_t)j]];
      } else {
        std::memset(dst, 0, rowb);
      }
    }
    g_err.clear();
    return SDNN_OK;
  }
  // global-tile path: live row i sits at position src[final_list][i] of the final tiles; rows are
  // gathered on the device into the other activation buffer (free after the run), in batches
  std::vector<int32_t> srcpos((size_t)std::max(c, 1));
  if (c > 0)
    HIP_OR_POISON(net, hipMemcpy(srcpos.data(), net->src[net->final_list], (size_t)c * sizeof(int32_t), hipMemcpyDeviceToHost));
  std::vector<int32_t> pos;
  std::vector<int64_t> which;
  for (int64_t q = 0; q < n; ++q) {
    float *dst = out_host + (size_t)q * net->N;
    std::memset(dst, 0, rowb);
    if (c == 0 || !net->final_fm) continue;
    auto it = std::lower_bound(live.begin(), live.begin() + c, (long long)ids[q]);
    if (it == live.begin() + c || *it != ids[q]) continue;
    pos.push_back(srcpos[(size_t)(it - live.begin())]);
    which.push_back(q);
  }
  float *stage = (net->final_fm == net->fm[0]) ? net->fm[1] : net->fm[0];
  int *dpos = net->ids[net->final_list ^ 1];
  const int64_t batch = std::max<int64_t>(1, net->M);
  for (size_t b0 = 0; b0 < pos.size(); b0 += (size_t)batch) {
    const int nb = (int)std::min<size_t>((size_t)batch, pos.size() - b0);
    HIP_OR_POISON(net, hipMemcpy(dpos, pos.data() + b0, (size_t)nb * sizeof(int32_t), hipMemcpyHostToDevice));
    const int64_t items = (int64_t)nb * net->N;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(net->cus * 8, (items + 255) / 256));
    hipLaunchKernelGGL(k_gather_rows, dim3(grid), dim3(256), 0, net->stream, net->final_fm, net->N, dpos, nb, stage);
    HIP_OR_POISON(net, hipGetLastError());
    HIP_OR_POISON(net, hipStreamSynchronize(net->stream));
    std::vector<float> rows((size_t)nb * net->N);
    HIP_OR_POISON(net, hipMemcpy(rows.data(), stage, (size_t)nb * rowb, hipMemcpyDeviceToHost));
    for (int i = 0; i < nb; ++i) {
      float *dst = out_host + (size_t)which[b0 + (size_t)i] * net->N;
      std::memcpy(dst, rows.data() + (size_t)i * net->N, rowb);
      // the last layer may have computed only one column of each group of equal columns
      if (!net->last_rep.empty())
        for (int32_t j = 0; j < net->N; ++j) dst[j] = dst[net->last_rep[(size_t)j]];
    }
  }
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_set_profiling(sdnn_net *net, int32_t enable) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (enable < 0 || enable > 2) return fail(SDNN_EINVAL, "profiling mode %d is not 0, 1 or 2", enable);
  net->pending_times = false;
  if (!enable) {
    net->profiling = false;
    g_err.clear();
    return SDNN_OK;
  }
  if (net->prof_start.empty()) {
    net->prof_start.resize((size_t)net->L);
    net->prof_end.resize((size_t)net->L);
    for (int32_t l = 0; l < net->L; ++l) {
      HIP_OR_POISON(net, hipEventCreate(&net->prof_start[(size_t)l]));
      HIP_OR_POISON(net, hipEventCreate(&net->prof_end[(size_t)l]));
    }
  }
  net->prof_ms.assign((size_t)net->L, 0.0);
  net->prof_runs.assign((size_t)net->L, 0);
  net->profiling = true;
  net->prof_mode = enable;
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_layer_info(sdnn_net *net, int32_t *kernel, int32_t *launches) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (!net->ran) return fail(SDNN_ESTATE, "no inference has run");
  if (!kernel || !launches) return fail(SDNN_EINVAL, "null array");
  for (int32_t l = 0; l < net->L; ++l) {
    kernel[l] = net->layer_kernel[(size_t)l];
    launches[l] = net->layer_launches[(size_t)l];
  }
  g_err.clear();
  return SDNN_OK;
}

sdnn_status sdnn_layer_times(sdnn_net *net, double *ms, int64_t *runs) {
  sdnn_status st = check_usable(net);
  if (st != SDNN_OK) return st;
  if (!ms || !runs) return fail(SDNN_EINVAL, "null array");
  for (int32_t l = 0; l < net->L; ++l) {
    ms[l] = net->prof_ms.empty() ? 0.0 : net->prof_ms[(size_t)l];
    runs[l] = net->prof_runs.empty() ? 0 : net->prof_runs[(size_t)l];
  }
  g_err.clear();
  return SDNN_OK;
}

void sdnn_destroy(sdnn_net *net) {
  if (!net) return;
  for (auto &ev : net->prof_start) (void)hipEventDestroy(ev);
  for (auto &ev : net->prof_end) (void)hipEventDestroy(ev);
  for (void *p : net->allocations) (void)hipFree(p);
  for (auto &ev : net->events) (void)hipEventDestroy(ev);
  if (net->pinned) (void)hipHostFree(net->pinned);
  if (net->progress) (void)hipHostFree(net->progress);
  if (net->notify) (void)hipHostFree(net->notify);
  delete net;
}

}  // extern "C"
