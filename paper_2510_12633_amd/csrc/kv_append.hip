// KV-cache append for paged decode on MI355X (gfx950).
//
// Each decode step writes the current token's key and value into its
// trajectory's last page before attention reads them (the KV cache of the
// paper's §5.2). One workgroup of two wavefronts per (trajectory, kv-head):
// wavefront 0 writes K, wavefront 1 writes V. The work is a few hundred
// bytes per unit, so the kernel is bound by launch and memory latency; it
// touches only the new token's slots, plus, for fp8 pages whose scale has
// to grow, the page's older codes.
//
// fp8 codes are OCP E4M3FN. Encoding is done in integer arithmetic on the
// fp32 bits (round to nearest, ties to even, after clamping to +-448), and
// decoding from the code fields, so the result depends on nothing but IEEE
// fp32 division and multiplication.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "laminar_kv_append.h"
#include "kv_append_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kFp8Max = 448.0f;

struct AppendArgs {
  const uint16_t* k_new;
  const uint16_t* v_new;
  int64_t row_stride;     // elements between trajectories' rows of k_new/v_new
  const int32_t* block_table;
  const int32_t* seq_lens;
  uint8_t* k_pages;
  uint8_t* v_pages;
  float* k_scale;
  float* v_scale;
  int32_t hkv, max_blocks, num_pages;
};

__device__ __forceinline__ float bf16_to_f32(uint32_t code) {
  return __uint_as_float(code << 16);
}

// |y| <= 448 -> E4M3FN code, round to nearest even; the sign bit follows y.
__device__ __forceinline__ uint32_t encode_e4m3fn(float y) {
  const uint32_t bits = __float_as_uint(y);
  const uint32_t sign = (bits >> 24) & 0x80u;
  const uint32_t a = bits & 0x7FFFFFFFu;
  uint32_t code;
  if (a < 0x3C800000u) {
    // below 2^-6 the codes are the multiples of 2^-9 (code 8 is 2^-6)
    code = uint32_t(__builtin_rintf(__uint_as_float(a) * 512.0f));
  } else {
    // keep 3 mantissa bits, rounding on the 20 dropped ones; a carry moves
    // into the exponent; rebias 127 -> 7
    code = ((a + 0x7FFFFu + ((a >> 20) & 1u)) >> 20) - (120u << 3);
  }
  return sign | code;
}

__device__ __forceinline__ float decode_e4m3fn(uint32_t code) {
  const uint32_t e = (code >> 3) & 0xFu, m = code & 7u;
  const float v = e ? __uint_as_float(((e + 120u) << 23) | (m << 20))
                    : float(m) * (1.0f / 512.0f);
  return (code & 0x80u) ? -v : v;
}

__device__ __forceinline__ uint32_t quantize(float x, float s) {
  return encode_e4m3fn(fminf(fmaxf(x / s, -kFp8Max), kFp8Max));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// New codes of dims 16c..16c+15 of the token (one K chunk), packed.
__device__ __forceinline__ u32x4 k_chunk_codes(const uint16_t* src, int c,
                                               float s) {
  const u32x4* s16 = reinterpret_cast<const u32x4*>(src) + 2 * c;
  const u32x4 lo = s16[0], hi = s16[1];
  u32x4 out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w0 = i < 2 ? lo[2 * i] : hi[2 * i - 4];
    const uint32_t w1 = i < 2 ? lo[2 * i + 1] : hi[2 * i - 3];
    out[i] = quantize(bf16_to_f32(w0 & 0xFFFFu), s) |
             quantize(bf16_to_f32(w0 >> 16), s) << 8 |
             quantize(bf16_to_f32(w1 & 0xFFFFu), s) << 16 |
             quantize(bf16_to_f32(w1 >> 16), s) << 24;
  }
  return out;
}

template <int D, bool FP8>
__global__ void __launch_bounds__(128) kv_append_kernel(const AppendArgs a) {
  const int unit = blockIdx.x;                      // b * hkv + kvh
  const int b = unit / a.hkv;
  const int kvh = unit - b * a.hkv;
  const bool is_v = (threadIdx.x >> 6) != 0;        // wave-uniform
  const int lane = threadIdx.x & 63;
  const uint16_t* src =
      (is_v ? a.v_new : a.k_new) + size_t(b) * a.row_stride + size_t(kvh) * D;
  // The new values do not depend on the table: load them first.
  constexpr int PER = D / 64;
  uint32_t xb[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) xb[i] = src[lane + 64 * i];

  const int n = a.seq_lens[b];
  if (n < 1) return;
  const int t = n - 1, blk = t >> 4, u = t & 15;
  if (blk >= a.max_blocks) return;
  const int pp = a.block_table[size_t(b) * a.max_blocks + blk];
  if (pp < 0 || pp >= a.num_pages) return;

  constexpr int EB = FP8 ? 1 : 2;
  constexpr int TILE = 16 * D * EB;                 // bytes per (page, head)
  uint8_t* tile = (is_v ? a.v_pages : a.k_pages) +
                  (size_t(pp) * a.hkv + kvh) * TILE;

  if constexpr (!FP8) {
    if (!is_v) {
      // K element (t, d) at ((d/8)*16 + t)*8 + d%8: 16-byte chunk c of the
      // token holds dims 8c..8c+7.
      if (lane < D / 8)
        reinterpret_cast<u32x4*>(tile)[lane * 16 + u] =
            reinterpret_cast<const u32x4*>(src)[lane];
    } else {
      // V element (t, d) at ((t/4)*D + d)*4 + t%4
      uint16_t* vt = reinterpret_cast<uint16_t*>(tile);
#pragma unroll
      for (int i = 0; i < PER; ++i)
        vt[((u >> 2) * D + lane + 64 * i) * 4 + (u & 3)] = uint16_t(xb[i]);
    }
    return;
  }

  // ---- fp8: the tile's scale, then the codes.
  float* scale = (is_v ? a.v_scale : a.k_scale) + size_t(pp) * a.hkv + kvh;
  const float s_old = *scale;                       // stale when u == 0
  // The lane's share of the old tile (16-byte vectors q = lane + 64 j),
  // read alongside the scale so that a re-encoding costs no extra trip.
  constexpr int NV = TILE / (64 * 16);
  u32x4 w[NV];
  if (u > 0) {
#pragma unroll
    for (int j = 0; j < NV; ++j)
      w[j] = reinterpret_cast<const u32x4*>(tile)[lane + 64 * j];
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) amax = fmaxf(amax, fabsf(bf16_to_f32(xb[i])));
  amax = wave_max(amax);
  const float c = amax / kFp8Max;

  // Token of byte k of vector q. K: a vector is one token's 16 dims (token
  // q % 16). V: a vector is 4 dims of token group q / (D/4), byte k being
  // token 4g + k%4 of dim 4 (q % (D/4)) + k/4.
  auto token = [&](int q, int k) {
    return is_v ? 4 * (q / (D / 4)) + (k & 3) : (q & 15);
  };
  bool any_old = false;
  if (u > 0 && s_old == 1.0f) {
#pragma unroll
    for (int j = 0; j < NV; ++j)
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const uint32_t code = (w[j][k >> 2] >> (8 * (k & 3))) & 0xFFu;
        any_old |= token(lane + 64 * j, k) < u && (code & 0x7Fu) != 0;
      }
  }
  any_old = __ballot(any_old) != 0;
  const bool empty = u == 0 || (s_old == 1.0f && !any_old);
  float s;
  bool recode = false;
  if (empty) {
    s = amax > 0.f ? c : 1.0f;
  } else if (c > s_old) {
    s = c;
    recode = true;
  } else {
    s = s_old;
  }
  if (lane == 0) *scale = s;

  if (recode) {                                     // wave-uniform
    // Every vector holding an old token is rewritten once, with the new
    // token's codes merged in where they share a vector, so no byte is
    // stored twice.
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int q = lane + 64 * j;
      u32x4 r = w[j];
      bool dirty = false;
      if (!is_v && token(q, 0) == u) {
        r = k_chunk_codes(src, q >> 4, s);
        dirty = true;
      } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int tok = token(q, k);
          const int sh = 8 * (k & 3);
          uint32_t nc;
          if (tok < u) {
            const uint32_t code = (r[k >> 2] >> sh) & 0xFFu;
            nc = quantize(decode_e4m3fn(code) * s_old, s);
          } else if (tok == u) {                    // V only
            const int d = 4 * (q % (D / 4)) + (k >> 2);
            nc = quantize(bf16_to_f32(src[d]), s);
          } else {
            continue;
          }
          r[k >> 2] = (r[k >> 2] & ~(0xFFu << sh)) | (nc << sh);
          dirty = true;
        }
      }
      if (dirty) reinterpret_cast<u32x4*>(tile)[q] = r;
    }
    return;
  }

  if (!is_v) {
    if (lane < D / 16)
      reinterpret_cast<u32x4*>(tile)[lane * 16 + u] = k_chunk_codes(src, lane, s);
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i)
      tile[((u >> 2) * D + lane + 64 * i) * 4 + (u & 3)] =
          uint8_t(quantize(bf16_to_f32(xb[i]), s));
  }
}

template <int D>
hipError_t launch(bool fp8, int units, const AppendArgs& a, hipStream_t st) {
  if (fp8)
    hipLaunchKernelGGL((kv_append_kernel<D, true>), dim3(units), dim3(128), 0,
                       st, a);
  else
    hipLaunchKernelGGL((kv_append_kernel<D, false>), dim3(units), dim3(128), 0,
                       st, a);
  return hipGetLastError();
}

}  // namespace

namespace laminar_detail {

laminar_status kv_append_check(const laminar_attn_desc* d, const void* k_new,
                               const void* v_new, const int32_t* block_table,
                               const int32_t* seq_lens, const void* k_pages,
                               const void* v_pages, const float* k_scale,
                               const float* v_scale, bool* empty) {
  *empty = false;
  if (!d || d->batch < 0 || d->num_kv_heads <= 0 || d->num_pages <= 0 ||
      d->max_blocks_per_seq < 0 || d->head_dim <= 0)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->kv_dtype != LAMINAR_KV_BF16 && d->kv_dtype != LAMINAR_KV_FP8_E4M3FN)
    return LAMINAR_ERR_INVALID_ARG;
  const bool fp8 = d->kv_dtype == LAMINAR_KV_FP8_E4M3FN;
  if (d->page_size != 16 || (d->head_dim != 64 && d->head_dim != 128))
    return LAMINAR_ERR_UNSUPPORTED;
  const int64_t units = int64_t(d->batch) * d->num_kv_heads;
  if (units > INT32_MAX) return LAMINAR_ERR_INVALID_ARG;
  if (units == 0) {
    *empty = true;
    return LAMINAR_OK;
  }
  if (!k_new || !v_new || !block_table || !seq_lens || !k_pages || !v_pages)
    return LAMINAR_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new) |
       reinterpret_cast<uintptr_t>(k_pages) |
       reinterpret_cast<uintptr_t>(v_pages)) & 15)
    return LAMINAR_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(block_table) |
       reinterpret_cast<uintptr_t>(seq_lens)) & 3)
    return LAMINAR_ERR_INVALID_ARG;
  if (fp8 && (!k_scale || !v_scale ||
              ((reinterpret_cast<uintptr_t>(k_scale) |
                reinterpret_cast<uintptr_t>(v_scale)) & 3)))
    return LAMINAR_ERR_INVALID_ARG;
  if (d->input_row_stride != 0 &&
      (int64_t(d->input_row_stride) < int64_t(d->num_kv_heads) * d->head_dim ||
       d->input_row_stride % 8 != 0))
    return LAMINAR_ERR_INVALID_ARG;
  return LAMINAR_OK;
}

}  // namespace laminar_detail

extern "C" laminar_status laminar_kv_append(
    const laminar_attn_desc* d, const void* k_new, const void* v_new,
    const int32_t* block_table, const int32_t* seq_lens, void* k_pages,
    void* v_pages, float* k_scale, float* v_scale, hipStream_t stream) {
  bool empty = false;
  const laminar_status st = laminar_detail::kv_append_check(
      d, k_new, v_new, block_table, seq_lens, k_pages, v_pages, k_scale,
      v_scale, &empty);
  if (st != LAMINAR_OK || empty) return st;
  const bool fp8 = d->kv_dtype == LAMINAR_KV_FP8_E4M3FN;
  const int64_t units = int64_t(d->batch) * d->num_kv_heads;
  AppendArgs a;
  a.row_stride = d->input_row_stride
                     ? d->input_row_stride
                     : int64_t(d->num_kv_heads) * d->head_dim;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.k_pages = static_cast<uint8_t*>(k_pages);
  a.v_pages = static_cast<uint8_t*>(v_pages);
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.hkv = d->num_kv_heads;
  a.max_blocks = d->max_blocks_per_seq;
  a.num_pages = d->num_pages;
  const hipError_t e = d->head_dim == 128
                           ? launch<128>(fp8, int(units), a, stream)
                           : launch<64>(fp8, int(units), a, stream);
  return e == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}
