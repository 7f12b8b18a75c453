// Skinny projection product y = x w^T for decode batches (M <= 128) on
// MI355X (gfx950).
//
// At decode batch sizes the product streams the whole weight matrix w
// [N, K] for a few rows of x, so it is bound by HBM bandwidth. The weights
// are packed once (laminar_linear_pack) into tiles of 16 rows whose 16-byte
// chunks (8 consecutive k of one row) are ordered (tile, k / 8, row): the
// 16 rows x 32 k that one v_mfma_f32_16x16x32_bf16 takes as its A operand
// are then 1 KB of contiguous bytes, and one load instruction of a
// wavefront reads exactly that.
//
// A workgroup is four wavefronts on four consecutive tiles (64 output
// features; eight tiles, two per wavefront, from 33 rows on) over one range
// of K. Per pipeline step of 128 k, each wavefront loads its tiles' 4 KB
// each of weights (non-temporal: they are read once) and
// the workgroup loads the batch's x [16 MT rows, 128 k] once and stages it
// in LDS, from where every wavefront reads its B operand; so x is fetched
// once per four tiles instead of once per tile (at M = 64 it would
// otherwise be four times the weight traffic). Four steps of loads are in
// flight (two from 33 rows on, whose tiles take more registers). All
// loads are buffer loads whose range check returns zeros: rows of x past
// M, the steps that pad the last group of NB, and a wavefront past the
// last tile read zeros without touching memory, so no load is conditional
// and the compiler keeps exact counts of the loads in flight.
// When N alone gives too few wavefronts to keep HBM busy, K is split and a
// second kernel adds the partial sums in a fixed order. For one to four
// rows and K up to 160 steps, the split stays inside a workgroup instead:
// its four wavefronts share one tile and take every fourth step, and their
// sums are added in LDS. That saves the second launch and the partial sums:
// 1-4 us of the 13-31 us that the QKV, O and down projections of 7B-32B
// models take at one row.
//
// When N / 128 groups of eight tiles leave the CUs unevenly loaded (the
// gate and up projection: 296 groups on 256 CUs left 40 CUs with twice the
// work), from 17 rows on a balanced split takes over: one workgroup of
// eight wavefronts per CU streams whole groups, then an equal share of the
// groups left over, cut along K; those pieces are added in a fixed order by
// a second kernel.
//
// x can also be what the decode step has at hand rather than the operand
// itself: the fp32 attention output, SwiGLU's gate and up, or the residual
// stream with an RMS norm in front (at most 8 rows). The staging makes the
// bf16 operand from it with the arithmetic of the separate kernel it
// replaces, and the K split does not depend on it, so the results are
// those of the separate launches bit for bit.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "activation.h"
#include "laminar_decode_step.h"
#include "kv_append_internal.h"
#include "laminar_linear.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStepK = 128;          // k values per pipeline step
constexpr int kMaxM = 128;
constexpr int kMaxK = 1 << 24;       // keeps weight offsets in 31 bits
// K is split into as many ranges as keep the grid within one workgroup per
// compute unit (256). Measured over the QKV, O and down projections of
// 7B-32B models at 1-128 rows, that beat two per CU by 3-13% at 5-32 rows
// and by up to 25% from 64 rows on (where the partial sums cost as much
// HBM traffic as the weights), and a third per CU lost 5-15% more.
constexpr int kMaxGroups = 256;
// the split inside one workgroup: at most 4 rows, 160 steps of K and 1024
// tiles (all workgroups resident at four per CU)
constexpr int kWaveSplitMaxM = 4;      // rows of the x layout in its LDS
constexpr int kWaveSplitMaxSteps = 160;
constexpr int kWaveSplitMaxTiles = 1024;
// Tiles per wavefront: from 33 rows on, each wavefront takes two tiles, so
// one staged x step feeds twice the weights (at M = 64 and 128 the QKV, O,
// down and LM-head products ran 10-17% faster than with one tile; gate+up
// was even).
template <int MT> constexpr int tiles_per_wave() { return MT >= 4 ? 2 : 1; }
// Steps in flight: 4 with one tile, 2 with two (registers).
template <int MT> constexpr int steps_in_flight() { return MT >= 4 ? 2 : 4; }
constexpr int kOob = 0x40000000;     // past every buffer: reads as zero
constexpr int kBufFlags = 0x00020000;

// What x holds: the bf16 operand itself, fp32 values rounded to bf16 on
// load, a SwiGLU's gate and up halves combined on load, or the input of an
// RMS norm (scaled by the row's 1 / rms and the norm weight on load).
constexpr int kXBf16 = 0, kXF32 = 1, kXSiluMul = 2, kXRmsNorm = 3;
// rows of the fused norm: one or two per wavefront of the workgroup
constexpr int kNormMaxM = 8;

struct LinearArgs {
  const void* x;         // [M, x_ld] of the kind the kernel is built for
  int32_t x_ld;          // elements per row of x: K, or 2 K for gate and up
  const uint16_t* norm_w;  // [K] bf16 weight of the fused RMS norm
  float norm_inv_k, norm_eps;
  const uint16_t* w;     // packed [N/16][K/8][16][8]
  float* y;              // [M, N] fp32 output, or NULL when yb is set
  uint16_t* yb;          // [M, N] bf16 output (rounded to nearest even)
  const uint16_t* res;   // [M, N] bf16 residual added before rounding, or NULL
  float* part;           // [splits, M, N] when split; balanced: [2 W, M, 128]
  int* counters;         // per group: pieces written so far (split only)
  int32_t m, n, k;
  int32_t n_tiles, splits, steps_per_split;
  // balanced split: each of W workgroups streams full_rounds whole groups
  // of eight tiles, then an equal share of the rem_groups left over
  int32_t wgs, full_rounds, rem_groups;
  // A step after the product that its reduction kernel makes when the call
  // has one: the RMS norm of each row of y (kPostNorm), or SwiGLU of y's
  // halves (kPostSwiGlu), into post_out.
  int32_t post_kind;
  const uint16_t* post_norm_w;   // [N] norm weight, or NULL
  float post_norm_inv_n, post_norm_eps;
  uint16_t* post_out;            // [M, N] or [M, N / 2] bf16
  // kPostAppend: the KV append of row m's new token (columns [k_col,
  // k_col + hkv D) and [v_col, ...) of y) into bf16 pools, as
  // laminar_kv_append stores it
  const int32_t* ap_lens;        // [M] lengths after the append
  const int32_t* ap_table;       // [M, max_blocks] block table
  uint16_t *ap_k, *ap_v;         // the K and V pools
  int32_t ap_k_col, ap_v_col, ap_hkv, ap_d, ap_max_blocks, ap_num_pages;
};

constexpr int kPostNone = 0, kPostNorm = 1, kPostSwiGlu = 2, kPostAppend = 3;

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// Final values of y[m, n .. n+3]: fp32, or bf16 of (value + residual).
__device__ __forceinline__ void store4(const LinearArgs& a, size_t off, f32x4 v) {
  if (!a.yb) {
    *reinterpret_cast<f32x4*>(a.y + off) = v;
    return;
  }
  if (a.res) {
    const bf16x4 r = *reinterpret_cast<const bf16x4*>(a.res + off);
    v += f32x4{float(r[0]), float(r[1]), float(r[2]), float(r[3])};
  }
  *reinterpret_cast<bf16x4*>(a.yb + off) =
      bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
}

// Waits for this wavefront's LDS writes, then for the whole workgroup; the
// loads in flight are not waited for (a plain __syncthreads would drain
// them). The empty asm statements keep the compiler from moving LDS
// accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0); vmcnt, expcnt free
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One 16-byte chunk of the bf16 operand (8 consecutive k of one row) as
// loaded: one load for bf16 x, two for fp32 x (32 bytes), for gate and up,
// or for x and the norm weight.
template <int XK> struct XRaw { u32x4 v[XK == kXBf16 ? 1 : 2]; };

template <int XK> constexpr int kXBytes = XK == kXF32 ? 4 : 2;

// Where x chunks come from: x itself, and the norm weight for kXRmsNorm.
struct XSource {
  __amdgpu_buffer_rsrc_t x, norm_w;
  int k_bytes;                  // gate to up, in bytes
};

XSource __device__ __forceinline__ x_source(const LinearArgs& a, int xe) {
  XSource src;
  src.x = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.x), 0,
                                            a.m * a.x_ld * xe, kBufFlags);
  src.norm_w = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.norm_w), 0, a.norm_w ? a.k * 2 : 0, kBufFlags);
  src.k_bytes = a.k * 2;
  return src;
}

// Loads the chunk at byte offset byte_off of x whose k is at byte offset
// k_off of a [K] bf16 row; offsets at or past kOob read zeros.
template <int XK>
__device__ __forceinline__ void load_x(XRaw<XK>& c, const XSource& src,
                                       int byte_off, int k_off) {
  c.v[0] = __builtin_bit_cast(
      u32x4, __builtin_amdgcn_raw_buffer_load_b128(src.x, byte_off, 0, 0));
  if constexpr (XK == kXF32)
    c.v[1] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(src.x, byte_off + 16, 0, 0));
  if constexpr (XK == kXSiluMul)     // up is K elements after gate
    c.v[1] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(src.x, byte_off + src.k_bytes,
                                                     0, 0));
  if constexpr (XK == kXRmsNorm)
    c.v[1] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(src.norm_w, k_off, 0, 0));
}

// The bf16 operand of a loaded chunk (zeros stay zeros in every kind; r is
// the row's 1 / rms for kXRmsNorm, 0 for rows past M).
template <int XK>
__device__ __forceinline__ u32x4 x_operand(const XRaw<XK>& c, float r) {
  if constexpr (XK == kXF32)
    return __builtin_bit_cast(
        u32x4, laminar::round8(__builtin_bit_cast(f32x4, c.v[0]),
                               __builtin_bit_cast(f32x4, c.v[1])));
  else if constexpr (XK == kXSiluMul)
    return __builtin_bit_cast(
        u32x4, laminar::silu_mul8(__builtin_bit_cast(bf16x8, c.v[0]),
                                  __builtin_bit_cast(bf16x8, c.v[1])));
  else if constexpr (XK == kXRmsNorm)
    return __builtin_bit_cast(
        u32x4, laminar::rms_scale8(__builtin_bit_cast(bf16x8, c.v[0]),
                                   __builtin_bit_cast(bf16x8, c.v[1]), r));
  else
    return c.v[0];
}

// 1 / rms of x row `row` (bf16, K per row), summed in laminar_rmsnorm's
// order: that kernel's thread t sums chunks t, t + 256, ... in one fma
// chain; here lane l of one wavefront keeps the chains of threads l,
// l + 64, l + 128 and l + 192, and each is added up by the same butterfly.
// 0 for rows past M.
__device__ __forceinline__ float row_rms_inverse(const LinearArgs& a,
                                                 __amdgpu_buffer_rsrc_t xr,
                                                 int row, int lane) {
  const int chunks = a.k >> 3;
  float p[4] = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < chunks; c0 += 256) {
    u32x4 v[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int c = c0 + 64 * b + lane;      // thread 64 b + lane
      v[b] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     xr, c < chunks ? (row * a.k + 8 * c) * 2 : kOob, 0, 0));
    }
#pragma unroll
    for (int b = 0; b < 4; ++b)
      p[b] = laminar::sumsq8(__builtin_bit_cast(bf16x8, v[b]), p[b]);
  }
#pragma unroll
  for (int w = 0; w < 4; ++w) p[w] = laminar::wave_sum(p[w]);
  const float r =
      laminar::rms_inverse(p[0], p[1], p[2], p[3], a.norm_inv_k, a.norm_eps);
  return row < a.m ? r : 0.f;
}

// Device-scope cache policy (SC1): a store with it is written through the
// XCD's L2 to memory, and a load with it is served from memory, not from a
// line a previous call left in the L2 -- the policy the compiler gives
// agent-scope atomic loads and stores. The partial sums of a K split take
// it both ways, so no L2 write-back or invalidation (a device-scope fence,
// about 30 us per call here) is needed to hand them between workgroups.
constexpr int kDevScope = 16;

// The partial sums of a K split as a buffer (at most 256 ranges x 128
// columns per group x 128 rows: far below 2 GiB).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t part_rsrc(const LinearArgs& a,
                                                            int pieces) {
  return __builtin_amdgcn_make_buffer_rsrc(
      a.part, 0, int(size_t(pieces) * a.m * a.n * sizeof(float)), kBufFlags);
}

// f32x4 store of a partial sum at float index off of a.part, device scope
__device__ __forceinline__ void store_part(__amdgpu_buffer_rsrc_t pr, size_t off,
                                           f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), pr,
                                         int(off * sizeof(float)), 0, kDevScope);
}

// Up to 32 rows, the last of a group's K ranges to finish adds them all (in
// range order) and writes the group's outputs, so no second kernel runs: at
// decode batch sizes each launch costs about 5 us, as much as the sum
// itself. (From 33 rows one workgroup reading every range of its group,
// 229 KB for 64 rows of QKV, took longer than linear_reduce, which spreads
// the sum over the GPU.) Each
// thread waits for its device-scope partial stores to complete before the
// workgroup counts its range in, with one atomic on the group's counter;
// the workgroup that completes the count reads every range with
// device-scope loads, and leaves the counter at zero for the next call.
// cols outputs per row from n0.
__device__ __forceinline__ void finish_group(const LinearArgs& a, int group,
                                             int pieces, int n0, int cols,
                                             int threads) {
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);          // this thread's stores are done
  __syncthreads();
  if (threadIdx.x == 0) {
    const int done = __hip_atomic_fetch_add(a.counters + group, 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = done == pieces - 1;
    if (done == pieces - 1)
      __hip_atomic_store(a.counters + group, 0, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!s_last) return;
  const size_t total = size_t(a.m) * a.n;
  const __amdgpu_buffer_rsrc_t pr = part_rsrc(a, pieces);
  const int c4n = cols / 4;
  for (int idx = threadIdx.x; idx < a.m * c4n; idx += threads) {
    const int m = idx / c4n;
    const int n = n0 + 4 * (idx - m * c4n);
    if (n >= a.n) continue;
    const size_t i = size_t(m) * a.n + n;
    f32x4 v[8];
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < pieces; k0 += 8) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        v[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                   pr, k0 + j < pieces ? int(((k0 + j) * total + i) * sizeof(float)) : kOob,
                   0, kDevScope));
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (k0 + j == 0) s = v[0];
        else if (k0 + j < pieces) s += v[j];
      }
    }
    store4(a, i, s);
  }
}

// y[m, n] = sum over splits s (in order) of part[s, m, n], then the output
// epilogue; four n per thread. Eight partial sums are loaded before the
// first add.
__global__ void __launch_bounds__(256) linear_reduce(const LinearArgs a) {
  const size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;    // float4 index
  const size_t total = size_t(a.m) * a.n / 4;
  if (i >= total) return;
  const f32x4* p = reinterpret_cast<const f32x4*>(a.part);
  f32x4 s = p[i];
  for (int k0 = 1; k0 < a.splits; k0 += 8) {
    f32x4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = k0 + j < a.splits ? p[size_t(k0 + j) * total + i]
                               : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k0 + j < a.splits) s += v[j];
  }
  store4(a, 4 * i, s);
}

// linear_reduce followed by the KV append of each row's new token: y as
// linear_reduce writes it, and where the four outputs are K or V of a
// kv-head, the same bf16 values stored at the token's slot of its page as
// laminar_kv_append stores them (K element (t, d) of a tile at
// ((d / 8) 16 + t) 8 + d % 8, V element at ((t / 4) D + d) 4 + t % 4). The
// token's length and block-table entry are loaded with the partial sums;
// nothing goes to the pools for a length below 1, a block past the table or
// a table entry outside the pool.
__global__ void __launch_bounds__(256) linear_reduce_append(const LinearArgs a) {
  const size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;    // float4 index
  const size_t total = size_t(a.m) * a.n / 4;
  if (i >= total) return;
  const int m = int(4 * i / size_t(a.n));
  const int n = int(4 * i - size_t(m) * a.n);
  const int hd = a.ap_hkv * a.ap_d;
  const bool is_k = n >= a.ap_k_col && n < a.ap_k_col + hd;
  const bool is_v = n >= a.ap_v_col && n < a.ap_v_col + hd;
  int page = -1, slot = 0;
  if (is_k || is_v) {
    const int len = a.ap_lens[m];
    const int t = len - 1;
    if (len >= 1 && (t >> 4) < a.ap_max_blocks) {
      const int e = a.ap_table[size_t(m) * a.ap_max_blocks + (t >> 4)];
      if (e >= 0 && e < a.ap_num_pages) {
        page = e;
        slot = t & 15;
      }
    }
  }
  const f32x4* p = reinterpret_cast<const f32x4*>(a.part);
  f32x4 s = p[i];
  for (int k0 = 1; k0 < a.splits; k0 += 8) {
    f32x4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      v[j] = k0 + j < a.splits ? p[size_t(k0 + j) * total + i]
                               : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k0 + j < a.splits) s += v[j];
  }
  store4(a, 4 * i, s);
  if (page < 0) return;
  // the values store4 wrote (one rounding; these calls have no residual)
  const bf16x4 o{(__bf16)s[0], (__bf16)s[1], (__bf16)s[2], (__bf16)s[3]};
  const int c = n - (is_k ? a.ap_k_col : a.ap_v_col);
  const int kvh = c / a.ap_d, d = c - kvh * a.ap_d;
  uint16_t* tile = (is_k ? a.ap_k : a.ap_v) +
                   (size_t(page) * a.ap_hkv + kvh) * 16 * a.ap_d;
  if (is_k) {
    *reinterpret_cast<bf16x4*>(tile + ((d >> 3) * 16 + slot) * 8 + (d & 7)) = o;
  } else {
    // the bits of the four values (a bit cast of one element of the bf16
    // vector read element 0 every time: cast the whole vector)
    typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
    const u16x4 ob = __builtin_bit_cast(u16x4, o);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      tile[((slot >> 2) * a.ap_d + d + e) * 4 + (slot & 3)] = ob[e];
  }
}

template <int MT, int XK>
__global__ void __launch_bounds__(256) linear_kernel(const LinearArgs a) {
  // x of one step, double-buffered: chunk (t, k/8 = c, row r) at
  // t * 256 + c * 16 + r, so the 64 lanes of a wavefront read 1 KB of
  // consecutive chunks for each matrix-core step
  __shared__ u32x4 xs[2][MT * 256];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  constexpr int TW = tiles_per_wave<MT>();
  const int tile0 = (blockIdx.x * 4 + wave) * TW;
  const int split = blockIdx.y;
  const int r16 = lane & 15, q = lane >> 4;
  const int total_steps = a.k / kStepK;
  const int s0 = split * a.steps_per_split;
  const int s1 = min(total_steps, s0 + a.steps_per_split);
  // this thread stages chunk (t, c = tid / 16, row tid % 16) of every step
  const int x_row = tid & 15, x_chunk = tid >> 4;

  // a wavefront past the last tile reads zeros
  __amdgpu_buffer_rsrc_t wr[TW];
#pragma unroll
  for (int tt = 0; tt < TW; ++tt) {
    const bool has = tile0 + tt < a.n_tiles;
    wr[tt] = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.w) + size_t(has ? tile0 + tt : 0) * 16 * a.k,
        0, has ? a.k * 32 : 0, kBufFlags);
  }
  constexpr int xe = kXBytes<XK>;
  const XSource xsrc = x_source(a, xe);
  // lane (q, r16) of matrix-core step j holds row r16, k chunk 4 j + q
  const int w_lane = (q * 16 + r16) * 16;

  constexpr int kNB = steps_in_flight<MT>();
  u32x4 wb[kNB][TW][4];
  XRaw<XK> xb[kNB][MT];
  auto load = [&](int s, int i) {
    const bool in = s < s1;
    const int kb = s * kStepK;
    const int wo = in ? kb * 32 + w_lane : kOob;
#pragma unroll
    for (int tt = 0; tt < TW; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        wb[i][tt][j] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       wr[tt], wo + 1024 * j, 0, /*nt*/ 2));
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int xo =
          in ? ((16 * t + x_row) * a.x_ld + kb + 8 * x_chunk) * xe : kOob;
      load_x<XK>(xb[i][t], xsrc, xo, in ? (kb + 8 * x_chunk) * 2 : kOob);
    }
  };

  f32x4 acc[TW][MT];
#pragma unroll
  for (int tt = 0; tt < TW; ++tt)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[tt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < kNB; ++i) load(s0 + i, i);
  // the fused norm (one tile of at most 8 rows): wavefront w finds the
  // 1 / rms of rows w and w + 4 while the first weights are on their way
  float r_row = 0.f;
  if constexpr (XK == kXRmsNorm) {
    static_assert(MT == 1, "the fused norm covers one 16-row tile");
    __shared__ float rr[kNormMaxM];
    const float r0 = row_rms_inverse(a, xsrc.x, wave, lane);
    const float r1 = a.m > 4 ? row_rms_inverse(a, xsrc.x, wave + 4, lane) : 0.f;
    if (lane == 0) {
      rr[wave] = r0;
      rr[wave + 4] = r1;
    }
    lds_barrier();
    r_row = x_row < kNormMaxM ? rr[x_row & 7] : 0.f;
  }
  // Steps past s1 (the last group padded to kNB steps) load zeros and add
  // nothing, so every step runs the same code.
  for (int st = s0; st < s1; st += kNB) {
#pragma unroll
    for (int i = 0; i < kNB; ++i) {
      const int s = st + i;
      u32x4* buf = xs[s & 1];
#pragma unroll
      for (int t = 0; t < MT; ++t) buf[t * 256 + tid] = x_operand<XK>(xb[i][t], r_row);
      // The buffer written here was last read two steps ago, before every
      // wavefront passed the previous step's barrier.
      lds_barrier();
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const bf16x8 bv =
              __builtin_bit_cast(bf16x8, buf[t * 256 + 64 * j + lane]);
#pragma unroll
          for (int tt = 0; tt < TW; ++tt)
            acc[tt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, wb[i][tt][j]), bv, acc[tt][t], 0,
                0, 0);
        }
      }
      load(s + kNB, i);
    }
  }

  // lane (group q, column r16) holds D[16 tile + 4q + r][m = 16t + r16]
  constexpr bool kFinishInKernel = MT <= 2;
  const __amdgpu_buffer_rsrc_t pr = part_rsrc(a, a.splits);
#pragma unroll
  for (int tt = 0; tt < TW; ++tt) {
    const int tile = tile0 + tt;
    if (tile >= a.n_tiles) break;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = 16 * t + r16;
      if (m >= a.m) continue;
      const size_t off = size_t(m) * a.n + tile * 16 + 4 * q;
      if (a.splits == 1)
        store4(a, off, acc[tt][t]);
      else if (kFinishInKernel)
        store_part(pr, size_t(split) * a.m * a.n + off, acc[tt][t]);
      else
        *reinterpret_cast<f32x4*>(a.part + size_t(split) * a.m * a.n + off) =
            acc[tt][t];
    }
  }
  if (kFinishInKernel && a.splits > 1)
    finish_group(a, blockIdx.x, a.splits, blockIdx.x * 64 * TW, 64 * TW, 256);
}


// ---------------------------------------------------------------------------
// Balanced split (from 17 rows, when the group grid is uneven). A workgroup
// is eight wavefronts on the eight tiles of a group (128 output features),
// one workgroup per CU (W = 256: its LDS use admits no second one). Each
// workgroup processes a stream of (group, step) units: first full_rounds
// whole groups (w, w + W, ...), whose sums are final, then its share
// [floor(w ru / W), floor((w + 1) ru / W)) of the ru = rem_groups x steps
// units left over, in (group, step) order: at most two pieces, whose
// partial sums go to slots 2 w and 2 w + 1 and are added by
// linear_balance_reduce in workgroup order. So every CU streams the same
// weight bytes, within one step.
// x of a step is staged in LDS row-major: row r's 16 chunks of 16 bytes
// (128 k) at slots r * 16 + (c ^ (r & 15)), so the 16 lanes of a
// matrix-core step that read chunk c of rows 0..15 meet no bank conflict,
// and one wavefront instruction moves 4 rows of x (4 x 256 contiguous
// bytes; the layout of linear_kernel read 16 rows x 64 bytes per
// instruction). bf16 x goes from memory into LDS directly (buffer load to
// LDS); the fused kinds are made in registers and written in the same
// layout, so every kind sums in the same order. x of a unit is loaded
// right after the unit's weights, NB units ahead: the vector-memory counter
// completes in order, so x loaded later than the weights in flight would
// make each wait for x drain them.
constexpr int kWideTiles = 8;
constexpr int kBalancedWgs = 256;
constexpr int kBalancedNB = 3;     // units in flight (x in LDS)
constexpr int kBalancedRegNB = 2;  // units in flight (x made in registers)

// s_waitcnt vmcnt(n); expcnt and lgkmcnt not waited for
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// First left-over unit of workgroup w: floor(w ru / W), W = 256 (a shift:
// the reductions evaluate it for every candidate piece of every output, and
// a division there cost more than the sums).
static_assert(kBalancedWgs == 256, "rem_start divides by 256 with a shift");
__host__ __device__ inline int64_t rem_start(int w, int64_t ru, int wgs) {
  (void)wgs;
  return (int64_t(w) * ru) >> 8;
}

// Position in a workgroup's stream of units.
struct UnitCursor {
  int g, s;        // group and step
  int round;       // full round, or full_rounds once in the left-over units
  int piece;       // left-over piece (0 or 1) of this workgroup
};

template <int MT, int XK, int NB, bool DMA>
__global__ void __launch_bounds__(512) linear_balanced_kernel(const LinearArgs a) {
  static_assert(MT >= 2 && XK != kXRmsNorm, "17 rows or more, no fused norm");
  static_assert(!DMA || XK == kXBf16, "only bf16 x is copied as it is");
  constexpr int NBUF = DMA ? NB + 1 : 2;
  constexpr int kBufSlots = MT * 256;
  constexpr int XPW = MT / 2;      // x instructions per wavefront and unit
  // more LDS than two workgroups could share: one workgroup per CU
  constexpr int kMinSlots = (81 * 1024) / 16;
  constexpr int kSlots = NBUF * kBufSlots > kMinSlots ? NBUF * kBufSlots : kMinSlots;
  __shared__ u32x4 xs[kSlots];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wg = blockIdx.x;
  const int W = a.wgs;
  const int r16 = lane & 15, q = lane >> 4;
  const int S = a.k / kStepK;
  const int gf = a.full_rounds * W;
  const int64_t ru = int64_t(a.rem_groups) * S;
  const int u0 = int(rem_start(wg, ru, W));
  const int u1 = int(rem_start(wg + 1, ru, W));
  const int n_units = a.full_rounds * S + (u1 - u0);
  constexpr int xe = kXBytes<XK>;
  const XSource xsrc = x_source(a, xe);
  const int w_lane = (q * 16 + r16) * 16;

  // rows past M stay zero (their loads read zeros or nothing)
  for (int i = tid; i < kSlots; i += 512) xs[i] = u32x4{0u, 0u, 0u, 0u};
  lds_barrier();

  auto start = [&](UnitCursor& c) {
    c.round = 0;
    c.piece = 0;
    if (a.full_rounds > 0) {
      c.g = wg;
      c.s = 0;
    } else {
      c.g = gf + u0 / S;
      c.s = u0 % S;
    }
  };
  auto advance = [&](UnitCursor& c) {
    if (++c.s < S) return;
    c.s = 0;
    if (c.round < a.full_rounds) {
      if (++c.round < a.full_rounds) {
        c.g += W;
      } else {
        c.g = gf + u0 / S;
        c.s = u0 % S;
      }
    } else {
      ++c.g;
      ++c.piece;
    }
  };

  u32x4 wb[NB][4];
  XRaw<XK> xr[DMA ? 1 : NB][XPW];
  UnitCursor lc;
  start(lc);
  int lv = 0;
  // loads unit lv (its weights, then its x) into set i; units past the
  // stream read zeros and are not computed
  auto issue = [&](int i) {
    const bool in = lv < n_units;
    const int tile = lc.g * kWideTiles + wave;
    const bool has = in && tile < a.n_tiles;
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.w) + size_t(has ? tile : 0) * 16 * a.k, 0,
        has ? a.k * 32 : 0, kBufFlags);
    const int wo = has ? lc.s * kStepK * 32 + w_lane : kOob;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      wb[i][j] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(wr, wo + 1024 * j, 0, /*nt*/ 2));
#pragma unroll
    for (int e = 0; e < XPW; ++e) {
      const int d = wave * XPW + e;              // rows 4d .. 4d + 3
      const int row = 4 * d + (lane >> 4);
      const int c = (lane & 15) ^ (row & 15);
      const bool inx = in && row < a.m;
      const int kb = lc.s * kStepK + 8 * c;
      const int off = inx ? (row * a.x_ld + kb) * xe : kOob;
      if constexpr (DMA) {
        u32x4* dst = xs + (lv % NBUF) * kBufSlots + d * 64;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            xsrc.x, (__attribute__((address_space(3))) void*)dst, 16, off, 0, 0, 0);
      } else {
        load_x<XK>(xr[i][e], xsrc, off, inx ? kb * 2 : kOob);
      }
    }
    ++lv;
    if (in) advance(lc);
  };

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  UnitCursor cc;
  start(cc);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    asm volatile("" ::: "memory");
    issue(i);
  }
  asm volatile("" ::: "memory");
  for (int v0 = 0; v0 < n_units; v0 += NB) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int v = v0 + i;
      const u32x4* buf;
      if constexpr (DMA) {
        // x of unit v went out (NB - 1) units of loads ago; stores issued
        // since only make this wait longer
        wait_vm<(NB - 1) * (4 + XPW)>();
        buf = xs + (v % NBUF) * kBufSlots;
      } else {
        // the buffer written here was last read two units ago, before
        // every wavefront passed the previous unit's barrier
        u32x4* wbuf = xs + (v & 1) * kBufSlots;
#pragma unroll
        for (int e = 0; e < XPW; ++e)
          wbuf[(wave * XPW + e) * 64 + lane] = x_operand<XK>(xr[i][e], 0.f);
        buf = wbuf;
      }
      lds_barrier();
      if (v < n_units) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            const int c = (4 * j + q) ^ r16;
            const bf16x8 bv = __builtin_bit_cast(bf16x8, buf[(16 * t + r16) * 16 + c]);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, wb[i][j]), bv, acc[t], 0, 0, 0);
          }
        }
        if (cc.s == S - 1 || v == n_units - 1) {
          // lane (q, r16) holds D[16 tile + 4q + r][m = 16t + r16]
          const int tile = cc.g * kWideTiles + wave;
          const bool whole = cc.round < a.full_rounds;
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            const int m = 16 * t + r16;
            if (m < a.m) {
              if (whole) {
                if (tile < a.n_tiles)
                  store4(a, size_t(m) * a.n + tile * 16 + 4 * q, acc[t]);
              } else {
                const size_t slot = size_t(2 * wg + cc.piece);
                *reinterpret_cast<f32x4*>(
                    a.part + (slot * a.m + m) * (kWideTiles * 16) + wave * 16 + 4 * q) =
                    acc[t];
              }
            }
            acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
        advance(cc);
      }
      asm volatile("" ::: "memory");
      issue(i);
      asm volatile("" ::: "memory");
    }
  }
  __builtin_amdgcn_s_waitcnt(0);     // no load into LDS outlives the workgroup
}

// Adds the pieces of each left-over group in workgroup order (the order of
// K), then the output epilogue; four outputs per thread. The pieces of a
// group come from consecutive workgroups; sixteen candidates (a group's
// pieces when W / rem_groups is at most 13) are loaded before the first
// add.
__global__ void __launch_bounds__(256) linear_balance_reduce(const LinearArgs a) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int per_group = a.m * (kWideTiles * 4);
  if (i >= int64_t(a.rem_groups) * per_group) return;
  const int rg = int(i / per_group);
  const int rem = int(i - int64_t(rg) * per_group);
  const int m = rem / (kWideTiles * 4), c4 = rem % (kWideTiles * 4);
  const int W = a.wgs, rgs = a.rem_groups;
  const int S = a.k / kStepK;
  const int n = (a.full_rounds * W + rg) * kWideTiles * 16 + 4 * c4;
  if (n >= a.n) return;
  const int64_t ru = int64_t(rgs) * S;
  const int64_t u = int64_t(rg) * S, u_end = u + S;
  const int w_lo = max(0, rg * W / rgs - 1);
  const int w_hi = min(W - 1, ((rg + 1) * W + rgs - 1) / rgs);
  f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
  int64_t s0 = rem_start(w_lo, ru, W);
  for (int w = w_lo; w <= w_hi; w += 16) {
    f32x4 v[16];
    bool use[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int ww = w + j;
      const int64_t s1 = rem_start(ww + 1, ru, W);
      // workgroup ww has units [s0, s1); group rg is its second piece when
      // its share began in the group before
      use[j] = ww <= w_hi && s1 > s0 && s0 < u_end && s1 > u;
      const size_t slot = size_t(2 * ww + (s0 < u ? 1 : 0));
      v[j] = use[j] ? *reinterpret_cast<const f32x4*>(
                          a.part + (slot * a.m + m) * (kWideTiles * 16) + 4 * c4)
                    : f32x4{0.f, 0.f, 0.f, 0.f};
      s0 = s1;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (use[j]) sum += v[j];
  }
  store4(a, size_t(m) * a.n + n, sum);
}

// Columns col .. col+7 of row m of a balanced call's bf16 output: read back
// when their group was whole (its workgroup wrote them), else the group's
// pieces added in workgroup order and rounded as linear_balance_reduce does
// (and written to y, which the call also returns).
__device__ __forceinline__ bf16x8 balanced_chunk8(const LinearArgs& a, int m, int col) {
  const int W = a.wgs;
  const int g = col / (kWideTiles * 16);
  const int gf = a.full_rounds * W;
  uint16_t* y8 = a.yb + size_t(m) * a.n + col;
  if (g < gf) return *reinterpret_cast<const bf16x8*>(y8);
  const int rg = g - gf, rgs = a.rem_groups;
  const int S = a.k / kStepK;
  const int64_t ru = int64_t(rgs) * S;
  const int64_t u = int64_t(rg) * S, u_end = u + S;
  const int w_lo = max(0, rg * W / rgs - 1);
  const int w_hi = min(W - 1, ((rg + 1) * W + rgs - 1) / rgs);
  const int c0 = col - g * kWideTiles * 16;
  f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = s0;
  int64_t st0 = rem_start(w_lo, ru, W);
  for (int w = w_lo; w <= w_hi; w += 8) {
    f32x4 v[8][2];
    bool use[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ww = w + j;
      const int64_t st1 = rem_start(ww + 1, ru, W);
      use[j] = ww <= w_hi && st1 > st0 && st0 < u_end && st1 > u;
      const size_t slot = size_t(2 * ww + (st0 < u ? 1 : 0));
      const float* q = a.part + (slot * a.m + m) * (kWideTiles * 16) + c0;
      v[j][0] = use[j] ? *reinterpret_cast<const f32x4*>(q) : f32x4{0.f, 0.f, 0.f, 0.f};
      v[j][1] = use[j] ? *reinterpret_cast<const f32x4*>(q + 4) : f32x4{0.f, 0.f, 0.f, 0.f};
      st0 = st1;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (use[j]) {
        s0 += v[j][0];
        s1 += v[j][1];
      }
  }
  const bf16x8 o{(__bf16)s0[0], (__bf16)s0[1], (__bf16)s0[2], (__bf16)s0[3],
                 (__bf16)s1[0], (__bf16)s1[1], (__bf16)s1[2], (__bf16)s1[3]};
  *reinterpret_cast<bf16x8*>(y8) = o;
  return o;
}

// The balanced split's reduction followed by SwiGLU of y's halves (gate
// columns 0 .. N/2 - 1, up columns N/2 ..): post_out exactly as
// laminar_silu_mul computes it from y, eight outputs per thread, in one
// launch instead of two.
__global__ void __launch_bounds__(256) linear_balance_reduce_swiglu(const LinearArgs a) {
  const int inter = a.n / 2, c8 = inter / 8;
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= int64_t(a.m) * c8) return;
  const int m = int(i / c8), j = int(i - int64_t(m) * c8) * 8;
  const bf16x8 g = balanced_chunk8(a, m, j);
  const bf16x8 u = balanced_chunk8(a, m, inter + j);
  *reinterpret_cast<bf16x8*>(a.post_out + size_t(m) * inter + j) = laminar::silu_mul8(g, u);
}

// One 16-row tile per workgroup, K split over its four wavefronts: wave w
// takes steps w, w + 4, w + 8, ... The sums of the four are added in LDS in
// wavefront order, so the result does not depend on timing. x has at most
// four rows here: per step a wavefront loads those rows' 128 k with one
// 16-byte chunk per lane (two for fp32 or gate and up), makes the bf16
// operand, and passes it through its own 1 KB of LDS into the matrix-core
// layout (rows 4-15 are zeros). So the raw x in flight takes 4-8 registers
// per step instead of the 16-32 of loading the operand layout directly.
template <int XK>
__global__ void __launch_bounds__(256) linear_wave_split_kernel(const LinearArgs a) {
  constexpr int kNB = 4;
  __shared__ f32x4 part[3][64];
  __shared__ u32x4 xw[4][64];          // per wavefront: x [4 rows][128 k]
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tile = blockIdx.x;
  const int r16 = lane & 15, q = lane >> 4;
  const int steps = a.k / kStepK;
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.w) + size_t(tile) * 16 * a.k, 0, a.k * 32,
      kBufFlags);
  constexpr int xe = kXBytes<XK>;
  const XSource xsrc = x_source(a, xe);
  const int w_lane = (q * 16 + r16) * 16;
  // this lane loads x row lane / 16, k chunk lane % 16 of each step, which
  // is chunk (lane / 16) * 16 + lane % 16 = lane of the wavefront's LDS
  const int x_lane = ((lane >> 4) * a.x_ld + 8 * (lane & 15)) * xe;
  u32x4 wb[kNB][4];
  XRaw<XK> xb[kNB];
  auto load = [&](int s, int i) {
    const bool in = s < steps;
    const int kb = s * kStepK;
    const int wo = in ? kb * 32 + w_lane : kOob;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      wb[i][j] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(wr, wo + 1024 * j, 0,
                                                       /*nt*/ 2));
    load_x<XK>(xb[i], xsrc, in ? kb * xe + x_lane : kOob,
               in ? (kb + 8 * (lane & 15)) * 2 : kOob);
  };
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4* xs = xw[wave];
#pragma unroll
  for (int i = 0; i < kNB; ++i) load(wave + 4 * i, i);
  // the fused norm (at most 4 rows here): wavefront w finds row w's 1 / rms
  // while the first weights are on their way; this lane's x row is lane / 16
  float r_row = 0.f;
  if constexpr (XK == kXRmsNorm) {
    __shared__ float rr[kNormMaxM];
    const float r = row_rms_inverse(a, xsrc.x, wave, lane);
    if (lane == 0) rr[wave] = r;
    lds_barrier();
    r_row = rr[lane >> 4];
  }
  for (int st = wave; st < steps; st += 4 * kNB) {
#pragma unroll
    for (int i = 0; i < kNB; ++i) {
      // LDS accesses of one wavefront complete in order: the reads below
      // see this write, and the next step's write follows these reads
      xs[lane] = x_operand<XK>(xb[i], r_row);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // lane (q, r16) of matrix-core step j: x row r16, k chunk 4 j + q
        const u32x4 xv = xs[(r16 & 3) * 16 + 4 * j + q];
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, wb[i][j]),
            __builtin_bit_cast(bf16x8, r16 < 4 ? xv : u32x4{0, 0, 0, 0}), acc,
            0, 0, 0);
      }
      load(st + 4 * i + 4 * kNB, i);
    }
  }
  if (wave > 0) part[wave - 1][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  acc += part[0][lane];
  acc += part[1][lane];
  acc += part[2][lane];
  if (r16 < a.m) store4(a, size_t(r16) * a.n + tile * 16 + 4 * q, acc);
}

// Columns 8c .. 8c+7 of row m as the group split's reduction writes them:
// the ranges added in order (all loads in flight first), then store4's
// epilogue (the residual, one rounding to bf16).
__device__ __forceinline__ bf16x8 reduce_chunk8(const LinearArgs& a, int m, int c) {
  const size_t total4 = size_t(a.m) * a.n / 4;
  const f32x4* p = reinterpret_cast<const f32x4*>(a.part);
  const size_t off = size_t(m) * a.n + 8 * c;
  const size_t i = off / 4;
  f32x4 s0 = p[i], s1 = p[i + 1];
  for (int k0 = 1; k0 < a.splits; k0 += 8) {
    f32x4 v[8][2];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = k0 + j < a.splits;
      v[j][0] = in ? p[size_t(k0 + j) * total4 + i] : f32x4{0.f, 0.f, 0.f, 0.f};
      v[j][1] = in ? p[size_t(k0 + j) * total4 + i + 1] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (k0 + j < a.splits) {
        s0 += v[j][0];
        s1 += v[j][1];
      }
  }
  if (a.res) {
    const bf16x4 r0 = *reinterpret_cast<const bf16x4*>(a.res + off);
    const bf16x4 r1 = *reinterpret_cast<const bf16x4*>(a.res + off + 4);
    s0 += f32x4{float(r0[0]), float(r0[1]), float(r0[2]), float(r0[3])};
    s1 += f32x4{float(r1[0]), float(r1[1]), float(r1[2]), float(r1[3])};
  }
  return bf16x8{(__bf16)s0[0], (__bf16)s0[1], (__bf16)s0[2], (__bf16)s0[3],
                (__bf16)s1[0], (__bf16)s1[1], (__bf16)s1[2], (__bf16)s1[3]};
}

// The group split's reduction for whole rows followed by the RMS norm of
// each row, one workgroup of 1024 threads per row: y exactly as
// linear_reduce writes it and post_out exactly as laminar_rmsnorm computes
// it from that y, in one launch instead of two. Thread t adds the ranges of
// chunk t (all loads of a row in one round: with 256 threads the row's
// 100-130 KB of partial sums took two); the row's chunks go through LDS so
// that threads 0-255 chain the sums of squares of chunks t, t + 256, ... in
// one fma each, then the same butterfly and sums, the same scaling and
// rounding as laminar_rmsnorm.
constexpr int kNormThreads = 1024;
constexpr int kNormMaxChunks = 2048;        // N up to 16384: 32 KB of LDS

__global__ void __launch_bounds__(kNormThreads) linear_reduce_norm(const LinearArgs a) {
  extern __shared__ bf16x8 yl[];            // the row's chunks of y
  __shared__ float part[4];
  const int m = blockIdx.x;
  const int chunks = a.n / 8;
  const int t = threadIdx.x;
  bf16x8* yr = reinterpret_cast<bf16x8*>(a.yb + size_t(m) * a.n);
  bf16x8* zr = reinterpret_cast<bf16x8*>(a.post_out + size_t(m) * a.n);
  const bf16x8* wr = reinterpret_cast<const bf16x8*>(a.post_norm_w);
  // the norm weight of the first chunk does not depend on the sums
  bf16x8 w0{};
  if (wr && t < chunks) w0 = wr[t];
  for (int c = t; c < chunks; c += kNormThreads) {
    const bf16x8 v = reduce_chunk8(a, m, c);
    yr[c] = v;
    yl[c] = v;
  }
  __syncthreads();
  if (t < 256) {
    float ss = 0.f;
    for (int c = t; c < chunks; c += 256) ss = laminar::sumsq8(yl[c], ss);
    ss = laminar::wave_sum(ss);
    if ((t & 63) == 0) part[t >> 6] = ss;
  }
  __syncthreads();
  const float r = laminar::rms_inverse(part[0], part[1], part[2], part[3],
                                       a.post_norm_inv_n, a.post_norm_eps);
  for (int c = t; c < chunks; c += kNormThreads) {
    const bf16x8 v = yl[c];
    if (wr) {
      zr[c] = laminar::rms_scale8(v, c == t ? w0 : wr[c], r);
    } else {
      bf16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (__bf16)(float(v[e]) * r);
      zr[c] = o;
    }
  }
}

// w [N, K] -> packed [N/16][K/8][16][8]: one 16-byte chunk per thread,
// indexed by its destination.
__global__ void __launch_bounds__(256)
pack_kernel(const u32x4* __restrict__ w, u32x4* __restrict__ out, int32_t n,
            int32_t k) {
  const size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;
  const size_t chunks = size_t(k) / 8;
  if (i >= size_t(n) * chunks) return;
  const size_t row = i & 15, rest = i >> 4;
  const size_t c = rest % chunks, tile = rest / chunks;
  out[i] = w[(tile * 16 + row) * chunks + c];
}

bool shape_ok(int32_t n, int32_t k) {
  return n >= 16 && n % 16 == 0 && k >= kStepK && k % kStepK == 0 &&
         k <= kMaxK;
}

bool shape_ok(int32_t m, int32_t n, int32_t k) {
  return m >= 1 && m <= kMaxM && shape_ok(n, k);
}

// Batch tiles of 16 rows the kernel is instantiated for: 1, 2, 4 or 8.
int launch_tiles(int32_t m) {
  const int mt = (m + 15) / 16;
  return mt <= 2 ? mt : (mt <= 4 ? 4 : 8);
}

struct SplitPlan {
  int32_t splits;      // K ranges over workgroups (1: none)
  int32_t per;         // steps per range
  bool wave_split;     // K split over the four wavefronts of a workgroup
};

// The K split over workgroups alone (what the workspace is sized for); a
// workgroup covers 4 tiles, or 8 from 33 rows on.
SplitPlan group_split_plan(int32_t m, int32_t n, int32_t k) {
  const int32_t tiles = n / 16, steps = k / kStepK;
  const int32_t per_group = launch_tiles(m) >= 4 ? 8 : 4;
  int32_t want = kMaxGroups / ((tiles + per_group - 1) / per_group);
  if (want < 1) want = 1;
  if (want > steps) want = steps;
  SplitPlan p;
  p.per = (steps + want - 1) / want;
  p.splits = (steps + p.per - 1) / p.per;
  p.wave_split = false;
  return p;
}

// The plan does not depend on what x holds, so the fused kinds of x sum in
// the same order as a bf16 x. A split over workgroups leaves at most 1024
// tiles, all resident with four workgroups per CU.
SplitPlan split_plan(int32_t m, int32_t n, int32_t k) {
  SplitPlan p = group_split_plan(m, n, k);
  const int32_t steps = k / kStepK;
  p.wave_split = m <= kWaveSplitMaxM && steps >= 2 &&
                 steps <= kWaveSplitMaxSteps && n / 16 <= kWaveSplitMaxTiles;
  if (p.wave_split) {
    p.splits = 1;
    p.per = steps;
  }
  return p;
}

struct BalancedPlan {
  bool use;
  int32_t wgs, full_rounds, rem_groups;
};

// The balanced split replaces the group grid from 17 rows on when that grid
// has more than 256 workgroups and its last round leaves the CUs uneven by
// more than 15% (rounds x 256 / workgroups; the pieces it cuts along K and
// their reduction cost a few microseconds, about what 15% of the gate and
// up projection is worth), and from 65 rows on whenever the grid has more
// than 256 workgroups: there its staging of x (whole rows, in LDS without
// registers, eight tiles per workgroup) also beat the group kernel on even
// grids (the 7B LM head at 128 rows: 236-260 us against 279-288).
BalancedPlan balanced_plan(int32_t m, int32_t n, int32_t k, const SplitPlan& sp) {
  BalancedPlan b{false, 0, 0, 0};
  const int32_t tiles = n / 16;
  if (sp.wave_split || launch_tiles(m) < 2) return b;
  const int32_t per_group = launch_tiles(m) >= 4 ? 8 : 4;
  const int64_t grid = int64_t((tiles + per_group - 1) / per_group) * sp.splits;
  if (grid <= kMaxGroups) return b;
  const int64_t rounds = (grid + kMaxGroups - 1) / kMaxGroups;
  if (launch_tiles(m) < 8 && rounds * kMaxGroups * 100 <= grid * 115) return b;
  const int32_t groups = (tiles + kWideTiles - 1) / kWideTiles;
  b.use = true;
  b.wgs = kBalancedWgs;
  b.full_rounds = groups / b.wgs;
  b.rem_groups = groups - b.full_rounds * b.wgs;
  return b;
}

// The most pieces any left-over group is cut into (1 when none is cut).
int32_t balanced_pieces(const BalancedPlan& b, int32_t k) {
  if (!b.rem_groups) return 1;
  const int64_t ru = int64_t(b.rem_groups) * (k / kStepK);
  int32_t most = 1;
  for (int rg = 0; rg < b.rem_groups; ++rg) {
    const int64_t u = int64_t(rg) * (k / kStepK), u_end = u + k / kStepK;
    int32_t count = 0;
    for (int w = 0; w < b.wgs; ++w) {
      const int64_t s0 = rem_start(w, ru, b.wgs), s1 = rem_start(w + 1, ru, b.wgs);
      if (s1 > s0 && s0 < u_end && s1 > u) ++count;
    }
    most = count > most ? count : most;
  }
  return most;
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// A workspace starts with one counter per group of a split that the last
// range of each group finishes (at most 256 groups), at the same place
// whatever the call's shape, so that calls of different M (or of different
// weights) can share one workspace: no call's partial sums cover another
// call's counters. The partial sums, or the balanced split's pieces, follow.
constexpr size_t kDataOffset = kMaxGroups * sizeof(int32_t);

size_t split_part_bytes(int32_t m, int32_t n, int32_t splits) {
  return align256(size_t(splits) * m * n * sizeof(float));
}

bool misaligned16(const void* p) {
  return reinterpret_cast<uintptr_t>(p) & 15;
}

}  // namespace

namespace {

template <int MT, int XK>
hipError_t launch_balanced(const LinearArgs& a, hipStream_t stream, bool& post_done) {
  const dim3 grid(a.wgs), block(512);
  if constexpr (XK == kXBf16)
    hipLaunchKernelGGL((linear_balanced_kernel<MT, XK, kBalancedNB, true>), grid,
                       block, 0, stream, a);
  else
    hipLaunchKernelGGL((linear_balanced_kernel<MT, XK, kBalancedRegNB, false>),
                       grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && a.rem_groups > 0) {
    if (a.post_kind == kPostSwiGlu) {
      const int64_t total = int64_t(a.m) * (a.n / 16);
      hipLaunchKernelGGL(linear_balance_reduce_swiglu,
                         dim3(unsigned((total + 255) / 256)), dim3(256), 0, stream, a);
      post_done = true;
    } else {
      const int64_t total = int64_t(a.rem_groups) * a.m * kWideTiles * 4;
      hipLaunchKernelGGL(linear_balance_reduce, dim3(unsigned((total + 255) / 256)),
                         dim3(256), 0, stream, a);
    }
    e = hipGetLastError();
  }
  return e;
}

template <int XK>
hipError_t launch(const LinearArgs& a, const SplitPlan& plan, bool balanced,
                  int m, hipStream_t stream, bool& post_done) {
  if constexpr (XK != kXRmsNorm) {
    if (balanced) {
      switch (launch_tiles(m)) {
        case 2: return launch_balanced<2, XK>(a, stream, post_done);
        case 4: return launch_balanced<4, XK>(a, stream, post_done);
        default: return launch_balanced<8, XK>(a, stream, post_done);
      }
    }
  }
  if (plan.wave_split) {
    hipLaunchKernelGGL((linear_wave_split_kernel<XK>), dim3(a.n_tiles),
                       dim3(256), 0, stream, a);
    return hipGetLastError();
  }
  // four wavefronts of tiles_per_wave tiles per workgroup
  const dim3 grid1((a.n_tiles + 3) / 4, a.splits);
  const dim3 grid2((a.n_tiles + 7) / 8, a.splits);
  if constexpr (XK == kXRmsNorm) {      // at most 8 rows: one tile
    hipLaunchKernelGGL((linear_kernel<1, XK>), grid1, dim3(256), 0, stream, a);
  } else {
    switch (launch_tiles(m)) {
      case 1: hipLaunchKernelGGL((linear_kernel<1, XK>), grid1, dim3(256), 0, stream, a); break;
      case 2: hipLaunchKernelGGL((linear_kernel<2, XK>), grid1, dim3(256), 0, stream, a); break;
      case 4: hipLaunchKernelGGL((linear_kernel<4, XK>), grid2, dim3(256), 0, stream, a); break;
      default: hipLaunchKernelGGL((linear_kernel<8, XK>), grid2, dim3(256), 0, stream, a); break;
    }
  }
  hipError_t e = hipGetLastError();
  // from 33 rows the partial sums are added by a second kernel, which also
  // makes the next RMS norm when the call asks for it
  if (e == hipSuccess && a.splits > 1 && launch_tiles(m) >= 4) {
    if (a.post_kind == kPostNorm && a.n / 8 <= kNormMaxChunks) {
      hipLaunchKernelGGL(linear_reduce_norm, dim3(unsigned(m)), dim3(kNormThreads),
                         size_t(a.n / 8) * sizeof(bf16x8), stream, a);
      post_done = true;
    } else if (a.post_kind == kPostAppend) {
      const size_t total = size_t(m) * a.n / 4;
      hipLaunchKernelGGL(linear_reduce_append, dim3(unsigned((total + 255) / 256)),
                         dim3(256), 0, stream, a);
      post_done = true;
    } else {
      const size_t total = size_t(m) * a.n / 4;
      hipLaunchKernelGGL(linear_reduce, dim3(unsigned((total + 255) / 256)),
                         dim3(256), 0, stream, a);
    }
    e = hipGetLastError();
  }
  return e;
}

// What follows the product in one call: nothing, the RMS norm of y, or
// SwiGLU of y's halves.
struct PostStep {
  int32_t kind = kPostNone;
  const void* norm_w = nullptr;   // RMS norm weight [N], or NULL
  float eps = 0.f;
  void* out = nullptr;            // [M, N] or [M, N / 2] bf16
  // kPostAppend: the append's description (input_row_stride N) and
  // arguments, checked by the caller
  const laminar_attn_desc* kv = nullptr;
  int32_t k_col = 0, v_col = 0;
  const int32_t* block_table = nullptr;
  const int32_t* seq_lens = nullptr;
  void *k_pages = nullptr, *v_pages = nullptr;
  float *k_scale = nullptr, *v_scale = nullptr;
};

laminar_status linear_impl(const void* x, int32_t x_kind, const void* w_packed,
                           float* y, void* yb, const void* res, int32_t m,
                           int32_t n, int32_t k, void* workspace,
                           size_t workspace_bytes, hipStream_t stream,
                           const void* norm_w = nullptr, float eps = 0.f,
                           const PostStep& post = PostStep()) {
  if (!x || !w_packed || (!y && !yb)) return LAMINAR_ERR_INVALID_ARG;
  if (x_kind != kXBf16 && x_kind != kXF32 && x_kind != kXSiluMul &&
      x_kind != kXRmsNorm)
    return LAMINAR_ERR_INVALID_ARG;
  if (misaligned16(x) || misaligned16(w_packed) || misaligned16(y) ||
      misaligned16(yb) || misaligned16(res) || misaligned16(norm_w))
    return LAMINAR_ERR_INVALID_ARG;
  if (x_kind == kXRmsNorm &&
      (!norm_w || !(eps >= 0.f) || !std::isfinite(eps)))
    return LAMINAR_ERR_INVALID_ARG;
  if (post.kind != kPostNone && post.kind != kPostAppend &&
      (!yb || !post.out || misaligned16(post.out) || misaligned16(post.norm_w) ||
       (post.kind == kPostNorm && (!(post.eps >= 0.f) || !std::isfinite(post.eps)))))
    return LAMINAR_ERR_INVALID_ARG;
  if (post.kind == kPostAppend && (!yb || !post.kv || res))
    return LAMINAR_ERR_INVALID_ARG;
  if (!shape_ok(m, n, k)) return LAMINAR_ERR_UNSUPPORTED;
  if (x_kind == kXRmsNorm && m > kNormMaxM) return LAMINAR_ERR_UNSUPPORTED;
  // byte offsets into x, padding rows included, stay below 2^31
  const size_t row_bytes = size_t(k) * (x_kind == kXBf16 ? 2 : 4);
  if (size_t(16) * launch_tiles(m) * row_bytes > size_t(kOob))
    return LAMINAR_ERR_UNSUPPORTED;
  LinearArgs a;
  a.x = x;
  a.x_ld = x_kind == kXSiluMul ? 2 * k : k;
  a.norm_w = static_cast<const uint16_t*>(norm_w);
  a.norm_inv_k = 1.0f / float(k);
  a.norm_eps = eps;
  a.w = static_cast<const uint16_t*>(w_packed);
  a.y = y;
  a.yb = static_cast<uint16_t*>(yb);
  a.res = static_cast<const uint16_t*>(res);
  a.m = m;
  a.n = n;
  a.k = k;
  a.n_tiles = n / 16;
  const SplitPlan plan = split_plan(m, n, k);
  const BalancedPlan bal = balanced_plan(m, n, k, plan);
  a.splits = bal.use ? 1 : plan.splits;
  a.steps_per_split = plan.per;
  a.wgs = bal.wgs;
  a.full_rounds = bal.full_rounds;
  a.rem_groups = bal.rem_groups;
  // the reduction stores bf16 K and V; fp8 pools take the append's own
  // launch (its per-page scales)
  const bool append_in_reduction =
      post.kind == kPostAppend && post.kv->kv_dtype == LAMINAR_KV_BF16 &&
      post.kv->batch > 0;
  a.post_kind = post.kind == kPostAppend && !append_in_reduction ? kPostNone
                                                                : post.kind;
  a.ap_lens = post.seq_lens;
  a.ap_table = post.block_table;
  a.ap_k = static_cast<uint16_t*>(post.k_pages);
  a.ap_v = static_cast<uint16_t*>(post.v_pages);
  a.ap_k_col = post.k_col;
  a.ap_v_col = post.v_col;
  a.ap_hkv = post.kv ? post.kv->num_kv_heads : 0;
  a.ap_d = post.kv ? post.kv->head_dim : 0;
  a.ap_max_blocks = post.kv ? post.kv->max_blocks_per_seq : 0;
  a.ap_num_pages = post.kv ? post.kv->num_pages : 0;
  a.post_norm_w = static_cast<const uint16_t*>(post.norm_w);
  a.post_norm_inv_n = 1.0f / float(n);
  a.post_norm_eps = post.eps;
  a.post_out = static_cast<uint16_t*>(post.out);
  a.part = nullptr;
  a.counters = nullptr;
  if (a.splits > 1 || (bal.use && bal.rem_groups > 0)) {
    const size_t need = laminar_linear_workspace_bytes(m, n, k);
    if (!workspace || workspace_bytes < need ||
        (reinterpret_cast<uintptr_t>(workspace) & 255))
      return LAMINAR_ERR_INVALID_ARG;
    a.counters = static_cast<int*>(workspace);
    a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) + kDataOffset);
  }
  hipError_t e;
  bool post_done = false;
  if (x_kind == kXF32)
    e = launch<kXF32>(a, plan, bal.use, m, stream, post_done);
  else if (x_kind == kXSiluMul)
    e = launch<kXSiluMul>(a, plan, bal.use, m, stream, post_done);
  else if (x_kind == kXRmsNorm)
    e = launch<kXRmsNorm>(a, plan, bal.use, m, stream, post_done);
  else
    e = launch<kXBf16>(a, plan, bal.use, m, stream, post_done);
  if (e != hipSuccess) return LAMINAR_ERR_HIP;
  // without a reduction kernel to carry it, the step is its own launch
  if (post.kind == kPostNorm && !post_done)
    return laminar_rmsnorm(yb, post.norm_w, post.out, m, n, post.eps, stream);
  if (post.kind == kPostSwiGlu && !post_done)
    return laminar_silu_mul(yb, post.out, m, n / 2, stream);
  if (post.kind == kPostAppend && !post_done) {
    uint16_t* y16 = static_cast<uint16_t*>(yb);
    return laminar_kv_append(post.kv, y16 + post.k_col, y16 + post.v_col,
                             post.block_table, post.seq_lens, post.k_pages,
                             post.v_pages, post.k_scale, post.v_scale, stream);
  }
  return LAMINAR_OK;
}

}  // namespace

extern "C" {

laminar_status laminar_linear_pack(const void* w, void* w_packed, int32_t n,
                                   int32_t k, hipStream_t stream) {
  if (!w || !w_packed || w == w_packed) return LAMINAR_ERR_INVALID_ARG;
  if (misaligned16(w) || misaligned16(w_packed)) return LAMINAR_ERR_INVALID_ARG;
  if (!shape_ok(n, k)) return LAMINAR_ERR_UNSUPPORTED;
  const size_t chunks = size_t(n) * k / 8;
  hipLaunchKernelGGL(pack_kernel, dim3(unsigned((chunks + 255) / 256)),
                     dim3(256), 0, stream, static_cast<const u32x4*>(w),
                     static_cast<u32x4*>(w_packed), n, k);
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

int32_t laminar_linear_splits(int32_t m, int32_t n, int32_t k) {
  if (!shape_ok(m, n, k)) return 0;
  const SplitPlan p = split_plan(m, n, k);
  const BalancedPlan b = balanced_plan(m, n, k, p);
  return b.use ? balanced_pieces(b, k) : p.splits;
}

size_t laminar_linear_workspace_bytes(int32_t m, int32_t n, int32_t k) {
  if (!shape_ok(m, n, k)) return 0;
  const SplitPlan p = split_plan(m, n, k);
  const BalancedPlan b = balanced_plan(m, n, k, p);
  if (b.use)
    return b.rem_groups ? kDataOffset + align256(size_t(2) * b.wgs * m * kWideTiles *
                                                 16 * sizeof(float))
                        : 0;
  return p.splits > 1 ? kDataOffset + split_part_bytes(m, n, p.splits) : 0;
}

laminar_status laminar_linear(const void* x, const void* w_packed, float* y,
                              int32_t m, int32_t n, int32_t k, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  if (!y) return LAMINAR_ERR_INVALID_ARG;
  return linear_impl(x, kXBf16, w_packed, y, nullptr, nullptr, m, n, k,
                     workspace, workspace_bytes, stream);
}

laminar_status laminar_linear_bf16(const void* x, const void* w_packed,
                                   void* y, const void* residual, int32_t m,
                                   int32_t n, int32_t k, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  if (!y) return LAMINAR_ERR_INVALID_ARG;
  return linear_impl(x, kXBf16, w_packed, nullptr, y, residual, m, n, k,
                     workspace, workspace_bytes, stream);
}

laminar_status laminar_linear_bf16_rmsnorm(const void* x,
                                           const void* norm_weight, float eps,
                                           const void* w_packed, void* y,
                                           const void* residual, int32_t m,
                                           int32_t n, int32_t k,
                                           void* workspace,
                                           size_t workspace_bytes,
                                           hipStream_t stream) {
  if (!y) return LAMINAR_ERR_INVALID_ARG;
  return linear_impl(x, kXRmsNorm, w_packed, nullptr, y, residual, m, n, k,
                     workspace, workspace_bytes, stream, norm_weight, eps);
}

laminar_status laminar_linear_bf16_norm(const void* x, int32_t x_kind,
                                        const void* w_packed, void* y,
                                        const void* residual,
                                        const void* norm_weight, float eps,
                                        void* y_norm, int32_t m, int32_t n,
                                        int32_t k, void* workspace,
                                        size_t workspace_bytes,
                                        hipStream_t stream) {
  if (!y || x_kind == kXRmsNorm) return LAMINAR_ERR_INVALID_ARG;
  PostStep post;
  post.kind = kPostNorm;
  post.norm_w = norm_weight;
  post.eps = eps;
  post.out = y_norm;
  return linear_impl(x, x_kind, w_packed, nullptr, y, residual, m, n, k,
                     workspace, workspace_bytes, stream, nullptr, 0.f, post);
}

laminar_status laminar_linear_bf16_swiglu(const void* x, int32_t x_kind,
                                          const void* w_packed, void* y,
                                          void* y_act, int32_t m, int32_t n,
                                          int32_t k, void* workspace,
                                          size_t workspace_bytes,
                                          hipStream_t stream) {
  if (!y || x_kind == kXRmsNorm) return LAMINAR_ERR_INVALID_ARG;
  PostStep post;
  post.kind = kPostSwiGlu;
  post.out = y_act;
  return linear_impl(x, x_kind, w_packed, nullptr, y, nullptr, m, n, k,
                     workspace, workspace_bytes, stream, nullptr, 0.f, post);
}

laminar_status laminar_linear_bf16_kv_append(
    const void* x, int32_t x_kind, const void* w_packed, void* y, int32_t m,
    int32_t n, int32_t k, void* workspace, size_t workspace_bytes,
    const laminar_attn_desc* kv_desc, int32_t k_col, int32_t v_col,
    const int32_t* block_table, const int32_t* seq_lens, void* k_pages,
    void* v_pages, float* k_scale, float* v_scale, hipStream_t stream) {
  if (!y || !kv_desc || x_kind == kXRmsNorm) return LAMINAR_ERR_INVALID_ARG;
  if (kv_desc->batch != m) return LAMINAR_ERR_INVALID_ARG;
  // the K and V columns: whole kv-heads inside y's rows, 16-byte aligned,
  // not overlapping
  const int64_t hd = int64_t(kv_desc->num_kv_heads) * kv_desc->head_dim;
  if (k_col < 0 || v_col < 0 || k_col % 8 || v_col % 8 || k_col + hd > n ||
      v_col + hd > n || (k_col < v_col + hd && v_col < k_col + hd))
    return LAMINAR_ERR_INVALID_ARG;
  laminar_attn_desc d = *kv_desc;
  d.input_row_stride = n;
  uint16_t* y16 = static_cast<uint16_t*>(y);
  bool empty = false;
  const laminar_status st = laminar_detail::kv_append_check(
      &d, y16 + k_col, y16 + v_col, block_table, seq_lens, k_pages, v_pages,
      k_scale, v_scale, &empty);
  if (st != LAMINAR_OK) return st;
  PostStep post;
  post.kind = kPostAppend;
  post.kv = &d;
  post.k_col = k_col;
  post.v_col = v_col;
  post.block_table = block_table;
  post.seq_lens = seq_lens;
  post.k_pages = k_pages;
  post.v_pages = v_pages;
  post.k_scale = k_scale;
  post.v_scale = v_scale;
  return linear_impl(x, x_kind, w_packed, nullptr, y, nullptr, m, n, k,
                     workspace, workspace_bytes, stream, nullptr, 0.f, post);
}

laminar_status laminar_linear_bf16_ex(const void* x, int32_t x_kind,
                                      const void* w_packed, void* y,
                                      const void* residual, int32_t m,
                                      int32_t n, int32_t k, void* workspace,
                                      size_t workspace_bytes,
                                      hipStream_t stream) {
  if (!y || x_kind == kXRmsNorm) return LAMINAR_ERR_INVALID_ARG;
  return linear_impl(x, x_kind, w_packed, nullptr, y, residual, m, n, k,
                     workspace, workspace_bytes, stream);
}

}  // extern "C"
