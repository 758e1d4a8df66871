// Span metadata, tied position ids, rotary embedding and decode-step commit.
//
// Span metadata follows Section 3.1 (sentinel tokens around a span; <CL>
// visible only to itself; enclosed tokens hidden from tokens after the <CR>)
// and the position tie of Section 3.1 "Input Transformation".
#include <math.h>

#include <cmath>
#include <cstring>
#include <vector>

#include "sckv_common.h"

namespace sckv {

// ---------------------------------------------------------------------------
// vu[t] and tied positions: one workgroup per sequence, 256 threads.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void span_meta_kernel(const int32_t* __restrict__ spans,
                                                        const int32_t* __restrict__ nspan,
                                                        int32_t b, int32_t s_max, int32_t L_meta,
                                                        int32_t* __restrict__ vu,
                                                        int32_t* __restrict__ pos) {
  const int s = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int32_t* cl = spans + (int64_t)s * s_max;
  const int32_t* cr = spans + (int64_t)b * s_max + (int64_t)s * s_max;
  const int n = nspan[s];
  __shared__ int wave_cnt[4];
  int carry = 0;
  for (int base = 0; base < L_meta; base += 256) {
    const int t = base + tid;
    bool normal = false;
    int v = SCKV_INF_VU;
    if (t < L_meta) {
      // last span whose <CL> is at or before t
      int lo = 0, hi = n;  // answer in [lo-1, hi-1]
      while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (cl[mid] <= t) lo = mid + 1; else hi = mid;
      }
      const int k = lo - 1;
      if (k >= 0 && t == cl[k]) {
        v = t;                          // <CL>
      } else if (k >= 0 && t < cr[k]) {
        v = cr[k];                      // enclosed token
        normal = true;
      } else if (k >= 0 && t == cr[k]) {
        v = SCKV_INF_VU;                // <CR>
      } else {
        normal = true;                  // plain normal token
      }
      vu[(int64_t)s * L_meta + t] = v;
    }
    const uint64_t m = __ballot(normal);
    const int rank = mask_rank(m);
    if ((tid & 63) == 0) wave_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = carry, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = wave_cnt[w];
      if (w < wave) off += c;
      total += c;
    }
    if (pos != nullptr && t < L_meta) {
      const int before = off + rank;  // normal tokens in [0, t)
      pos[(int64_t)s * L_meta + t] = normal ? before : (before > 0 ? before - 1 : 0);
    }
    carry += total;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// rotary embedding, rotate-half form: pair (i, i + d/2) turns by
// pos * theta^(-2i/d).  A thread owns one 16-byte piece of the first half of
// one token's rows (and the matching piece of the second half) in a group of
// hpt heads: it takes the piece's angles once and applies them to the
// token's row in each head of the group, so the group shares the sines and
// cosines.
// ---------------------------------------------------------------------------
struct InvFreq {
  double w[64];
};
// heads per thread of a rotation: two halves the angle work and keeps
// enough threads in flight (measured faster than 4..32 on 16x32x4096x80)
constexpr int ROPE_HPT = 2;

// row0 (nullable): per sequence, the row of y that receives row 0 of x; a
// sequence whose rows would leave [0, y_rows) (row0 < 0 included) is not
// written and sets SCKV_STATUS_CAP.
template <typename T, int D>
__global__ __launch_bounds__(256) void rope_kernel(const T* x, T* y,
                                                   int32_t b, int32_t H, int32_t n, int64_t xs,
                                                   int64_t ys, const int32_t* __restrict__ pos,
                                                   int32_t L_meta, int32_t tok0, InvFreq inv,
                                                   int rotate, int32_t hpt,
                                                   const int32_t* __restrict__ row0,
                                                   int32_t y_rows, int32_t* status) {
  constexpr int E = Piece<T>::E;
  constexpr int HALF = D / 2;
  constexpr int PPH = HALF / E;  // pieces per half row
  static_assert(HALF % E == 0, "half row must be whole pieces");
  const double two_pi = 6.283185307179586476925286766559;
  const int g = blockIdx.x * blockDim.x + threadIdx.x;  // (token, piece) of a sequence
  const int t = g / PPH;
  const int p = g - t * PPH;
  if (t >= n) return;
  // the piece's inverse frequencies, picked from the argument table
  double w[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    w[e] = 0.0;
#pragma unroll
    for (int pp = 0; pp < PPH; ++pp) w[e] = p == pp ? inv.w[pp * E + e] : w[e];
  }
  const int n_hg = (H + hpt - 1) / hpt;
  for (int sg = blockIdx.y; sg < b * n_hg; sg += gridDim.y) {
    const int s = sg / n_hg;
    const int h0 = (sg - s * n_hg) * hpt;
    const int h1 = min(h0 + hpt, H);
    int64_t drow = t;
    if (row0) {
      const int r0 = row0[s];
      if (r0 < 0 || (int64_t)r0 + n > y_rows) {
        if (status && g == 0 && h0 == 0) atomicOr(status, SCKV_STATUS_CAP);
        continue;
      }
      drow += r0;
    }
    float cs[E], sn[E];
    if (rotate) {
      const double ps = (double)pos[(int64_t)s * L_meta + tok0 + t];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        double ang = ps * w[e];
        ang -= two_pi * rint(ang / two_pi);
        sincosf((float)ang, &sn[e], &cs[e]);
      }
    }
    const T* src = x + (int64_t)s * H * xs + (int64_t)t * D + p * E;
    T* dst = y + (int64_t)s * H * ys + drow * D + p * E;
#pragma unroll 4
    for (int h = h0; h < h1; ++h) {
      u32x4 a = ld16(src + h * xs), c = ld16(src + h * xs + HALF);
      if (rotate) {
        float fa[E], fc[E];
        Piece<T>::unpack(a, fa);
        Piece<T>::unpack(c, fc);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float x1 = fa[e], x2 = fc[e];
          fa[e] = x1 * cs[e] - x2 * sn[e];
          fc[e] = x2 * cs[e] + x1 * sn[e];
        }
        a = Piece<T>::pack(fa);
        c = Piece<T>::pack(fc);
      }
      st16(dst + h * ys, a);
      st16(dst + h * ys + HALF, c);
    }
  }
}

// ---------------------------------------------------------------------------
// decode-step commit: one thread per sequence
// ---------------------------------------------------------------------------
__global__ void commit_kernel(int32_t* __restrict__ kv_len, int32_t* __restrict__ tok_idx,
                              int32_t* __restrict__ pos_ids, int32_t* __restrict__ cur_tok,
                              const int32_t* __restrict__ vu, const int32_t* __restrict__ pos,
                              int32_t L_meta, int32_t b, int32_t L_cap, int32_t* status) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= b) return;
  const int t = cur_tok[s];
  if (t < 0 || t >= L_meta) {
    if (status) atomicOr(status, SCKV_STATUS_TOKEN);
  } else if (vu[(int64_t)s * L_meta + t] != t) {
    const int n = kv_len[s];
    if (n < 0 || n >= L_cap) {
      if (status) atomicOr(status, SCKV_STATUS_CAP);
    } else {
      tok_idx[(int64_t)s * L_cap + n] = t;
      pos_ids[(int64_t)s * L_cap + n] = pos[(int64_t)s * L_meta + t];
      kv_len[s] = n + 1;
    }
  }
  cur_tok[s] = t + 1;
}

// ---------------------------------------------------------------------------
// block append bookkeeping: one workgroup per sequence
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void extend_kernel(int32_t* __restrict__ kv_len,
                                                     int32_t* __restrict__ tok_idx,
                                                     int32_t* __restrict__ pos_ids,
                                                     int32_t* __restrict__ row0_out,
                                                     const int32_t* __restrict__ pos,
                                                     int32_t L_meta, int32_t tok0, int32_t n,
                                                     int32_t L_cap, int32_t* status) {
  const int s = blockIdx.x;
  const int r0 = kv_len[s];
  const bool ok = r0 >= 0 && (int64_t)r0 + n <= L_cap;
  if (ok) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      tok_idx[(int64_t)s * L_cap + r0 + i] = tok0 + i;
      pos_ids[(int64_t)s * L_cap + r0 + i] = pos[(int64_t)s * L_meta + tok0 + i];
    }
  }
  __syncthreads();  // every thread has read kv_len[s]
  if (threadIdx.x == 0) {
    row0_out[s] = ok ? r0 : -1;
    if (ok) kv_len[s] = r0 + n;
    else if (status) atomicOr(status, SCKV_STATUS_CAP);
  }
}

}  // namespace sckv

using namespace sckv;

extern "C" int sckv_span_meta(const int32_t* cl_host, const int32_t* cr_host,
                              const int32_t* n_host, int32_t s_max, int32_t b, int32_t L_meta,
                              int32_t* spans_dev, int32_t* vu, int32_t* pos, hipStream_t stream) {
  clear_error();
  if (!cl_host || !cr_host || !n_host || !spans_dev || !vu)
    return fail(SCKV_EINVAL, "sckv_span_meta: null pointer");
  if (b <= 0 || s_max <= 0 || L_meta <= 0)
    return fail(SCKV_EINVAL, "sckv_span_meta: b, s_max and L_meta must be positive");
  for (int s = 0; s < b; ++s) {
    const int n = n_host[s];
    if (n < 0 || n > s_max)
      return fail(SCKV_ESPAN, "sckv_span_meta: span count of sequence " + std::to_string(s) +
                                  " outside [0, s_max]");
    for (int k = 0; k < n; ++k) {
      const int32_t c = cl_host[(int64_t)s * s_max + k], r = cr_host[(int64_t)s * s_max + k];
      if (c < 0 || c >= L_meta || r <= c)
        return fail(SCKV_ESPAN, "sckv_span_meta: sequence " + std::to_string(s) + " span " +
                                    std::to_string(k) + " needs 0 <= cl < L_meta and cl < cr");
      if (k > 0 && c <= cr_host[(int64_t)s * s_max + k - 1])
        return fail(SCKV_ESPAN, "sckv_span_meta: sequence " + std::to_string(s) + " span " +
                                    std::to_string(k) + " overlaps or is out of order");
    }
  }
  // Pack [cl | cr | n] and copy it in one transfer.  The source is a
  // pageable host vector: the copy has consumed it when the call returns.
  std::vector<int32_t> packed((size_t)2 * b * s_max + b);
  std::memcpy(packed.data(), cl_host, (size_t)b * s_max * sizeof(int32_t));
  std::memcpy(packed.data() + (size_t)b * s_max, cr_host, (size_t)b * s_max * sizeof(int32_t));
  std::memcpy(packed.data() + (size_t)2 * b * s_max, n_host, (size_t)b * sizeof(int32_t));
  int rc = hip_check(hipMemcpyAsync(spans_dev, packed.data(), packed.size() * sizeof(int32_t),
                                    hipMemcpyHostToDevice, stream),
                     "sckv_span_meta: span upload");
  if (rc) return rc;
  span_meta_kernel<<<b, 256, 0, stream>>>(spans_dev, spans_dev + (size_t)2 * b * s_max, b, s_max,
                                          L_meta, vu, pos);
  return hip_check(hipGetLastError(), "sckv_span_meta: launch");
}

template <typename T, int D>
static int launch_rope(const void* x, void* y, int32_t b, int32_t H, int32_t n, int64_t xs,
                       int64_t ys, const int32_t* pos, int32_t L_meta, int32_t tok0, float theta,
                       const int32_t* row0, int32_t y_rows, int32_t* status,
                       hipStream_t stream) {
  InvFreq inv;
  for (int i = 0; i < 64; ++i) inv.w[i] = 0.0;
  for (int i = 0; i < D / 2; ++i) inv.w[i] = std::pow((double)theta, -2.0 * i / D);
  constexpr int PPH = D / 2 / Piece<T>::E;
  const int64_t per_seq = (int64_t)n * PPH;
  if (per_seq > 0x7fffffffLL - 255) return fail(SCKV_EUNSUP, "rope_apply: too many rows");
  // heads per thread: a rotation shares its angles over ROPE_HPT heads; a
  // plain copy takes one head per thread
  const int rotate = theta > 0.f ? 1 : 0;
  const int hpt = rotate ? (H < ROPE_HPT ? H : ROPE_HPT) : 1;
  const int64_t groups = (int64_t)b * ((H + hpt - 1) / hpt);
  const dim3 grid((unsigned)((per_seq + 255) / 256), (unsigned)(groups < 65535 ? groups : 65535));
  rope_kernel<T, D><<<grid, 256, 0, stream>>>(
      static_cast<const T*>(x), static_cast<T*>(y), b, H, n, xs, ys, pos, L_meta, tok0, inv,
      rotate, hpt, row0, y_rows, status);
  return hip_check(hipGetLastError(), "rope_apply: launch");
}

static int rope_common(const char* who, const void* x, void* y, int32_t b, int32_t H, int32_t n,
                       int64_t x_stride_bh, int64_t y_stride_bh, int32_t d_head, sckv_dtype dt,
                       const int32_t* pos, int32_t L_meta, int32_t tok0, float theta,
                       const int32_t* row0, int32_t y_rows, int32_t* status, hipStream_t stream) {
  const std::string w(who);
  if (!x || !y) return fail(SCKV_EINVAL, w + ": null pointer");
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, w + ": unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, w + ": d_head must be 64 or 80");
  if (b <= 0 || H <= 0 || n < 0) return fail(SCKV_EINVAL, w + ": bad sizes");
  if (x_stride_bh < (int64_t)n * d_head)
    return fail(SCKV_EINVAL, w + ": x slice stride smaller than n*d_head");
  if (row0 ? (y_rows < n || y_stride_bh < (int64_t)y_rows * d_head)
           : y_stride_bh < (int64_t)n * d_head)
    return fail(SCKV_EINVAL, w + ": y slice smaller than its rows");
  if (!(theta >= 0.f) || std::isinf(theta)) return fail(SCKV_EINVAL, w + ": theta must be finite and >= 0");
  if (theta > 0.f) {
    if (!pos) return fail(SCKV_EINVAL, w + ": null pos");
    if (tok0 < 0 || L_meta <= 0 || (int64_t)tok0 + n > L_meta)
      return fail(SCKV_EINVAL, w + ": rows [tok0, tok0+n) exceed L_meta");
  }
  if (!aligned16(x) || !aligned16(y) || (x_stride_bh * elem_bytes(dt)) % 16 ||
      (y_stride_bh * elem_bytes(dt)) % 16)
    return fail(SCKV_EINVAL, w + ": buffers and strides must be 16-byte aligned");
  if (n == 0) return SCKV_OK;
  if (dt == SCKV_BF16)
    return d_head == 64 ? launch_rope<uint16_t, 64>(x, y, b, H, n, x_stride_bh, y_stride_bh, pos, L_meta, tok0, theta, row0, y_rows, status, stream)
                        : launch_rope<uint16_t, 80>(x, y, b, H, n, x_stride_bh, y_stride_bh, pos, L_meta, tok0, theta, row0, y_rows, status, stream);
  return d_head == 64 ? launch_rope<float, 64>(x, y, b, H, n, x_stride_bh, y_stride_bh, pos, L_meta, tok0, theta, row0, y_rows, status, stream)
                      : launch_rope<float, 80>(x, y, b, H, n, x_stride_bh, y_stride_bh, pos, L_meta, tok0, theta, row0, y_rows, status, stream);
}

extern "C" int rope_apply(const void* x, void* y, int32_t b, int32_t H, int32_t n,
                          int64_t x_stride_bh, int64_t y_stride_bh, int32_t d_head, sckv_dtype dt,
                          const int32_t* pos, int32_t L_meta, int32_t tok0, float theta,
                          hipStream_t stream) {
  clear_error();
  return rope_common("rope_apply", x, y, b, H, n, x_stride_bh, y_stride_bh, d_head, dt, pos,
                     L_meta, tok0, theta, nullptr, 0, nullptr, stream);
}

extern "C" int rope_apply_at(const void* x, void* y, const int32_t* row0, int32_t y_rows,
                             int32_t b, int32_t H, int32_t n, int64_t x_stride_bh,
                             int64_t y_stride_bh, int32_t d_head, sckv_dtype dt,
                             const int32_t* pos, int32_t L_meta, int32_t tok0, float theta,
                             int32_t* status, hipStream_t stream) {
  clear_error();
  if (!row0) return fail(SCKV_EINVAL, "rope_apply_at: null row0");
  return rope_common("rope_apply_at", x, y, b, H, n, x_stride_bh, y_stride_bh, d_head, dt, pos,
                     L_meta, tok0, theta, row0, y_rows, status, stream);
}

extern "C" int kv_extend(int32_t* kv_len, int32_t* tok_idx, int32_t* pos_ids, int32_t* row0_out,
                         const int32_t* pos, int32_t L_meta, int32_t tok0, int32_t n, int32_t b,
                         int32_t L_cap, int32_t* status, hipStream_t stream) {
  clear_error();
  if (!kv_len || !tok_idx || !pos_ids || !row0_out || !pos)
    return fail(SCKV_EINVAL, "kv_extend: null pointer");
  if (b <= 0 || L_cap <= 0 || L_meta <= 0 || n < 0) return fail(SCKV_EINVAL, "kv_extend: bad sizes");
  if (tok0 < 0 || (int64_t)tok0 + n > L_meta)
    return fail(SCKV_EINVAL, "kv_extend: tokens [tok0, tok0+n) exceed L_meta");
  extend_kernel<<<b, 256, 0, stream>>>(kv_len, tok_idx, pos_ids, row0_out, pos, L_meta, tok0, n,
                                       L_cap, status);
  return hip_check(hipGetLastError(), "kv_extend: launch");
}

extern "C" int kv_commit(int32_t* kv_len, int32_t* tok_idx, int32_t* pos_ids, int32_t* cur_tok,
                         const int32_t* vu, const int32_t* pos, int32_t L_meta, int32_t b,
                         int32_t L_cap, int32_t* status, hipStream_t stream) {
  clear_error();
  if (!kv_len || !tok_idx || !pos_ids || !cur_tok || !vu || !pos)
    return fail(SCKV_EINVAL, "kv_commit: null pointer");
  if (b <= 0 || L_cap <= 0 || L_meta <= 0) return fail(SCKV_EINVAL, "kv_commit: bad sizes");
  commit_kernel<<<(b + 255) / 256, 256, 0, stream>>>(kv_len, tok_idx, pos_ids, cur_tok, vu, pos,
                                                     L_meta, b, L_cap, status);
  return hip_check(hipGetLastError(), "kv_commit: launch");
}
