// One decode step over the compacted cache, split over key chunks.
// Section 1 and Section 2 (the key/value memory read per step drives decode
// cost) and Section 4.3 (generation continues from the compressed cache).
//
// decode_chunk_kernel : one workgroup per (sequence, head, chunk of CH rows),
//   chunk-major (chunks of one slice share no data but q, so L2 placement
//   does not matter; idle workgroups past a slice's end go last).  A
//   workgroup streams its rows with a 16-byte piece per lane; a row is spread
//   over LPR lanes of an aligned power-of-two group of GRP lanes, so the row
//   dot product is a DPP butterfly inside the group.  Each lane group keeps an
//   online softmax; the groups of the workgroup are merged through LDS into
//   one partial (max, sum, unnormalised output) in log2 units.  The
//   workgroup whose chunk holds row kv_len also rotates the new key and writes
//   the new key/value pair there.
// decode_combine_kernel : merges the partials of each slice (log-sum-exp) and
//   writes the output; a <CL> step outputs v_new, a failed step NaN.  Being a
//   separate launch on the same stream, it sees every partial without any
//   device-wide cache flush inside the chunk kernel.
#include <math.h>

#include <cmath>

#include "sckv_common.h"

namespace sckv {

// Tuning (measured on MI355X over the OPT-1.3B, 3B-RoPE and batch-256
// streaming decode shapes): 1024-row chunks, 4 rows per lane group in flight
// per trip, 256 threads, chunk-major dispatch order.
constexpr int DEC_THREADS = 256;
constexpr int DEC_CH = 1024;  // rows per chunk (one workgroup)
constexpr float LOG2E = 1.4426950408889634f;

struct RopeTab {
  double w[40];  // theta^(-2i/d), i < d/2
};

template <typename T, int D>
struct DecCfg {
  static constexpr int E = Piece<T>::E;           // elements per piece
  static constexpr int LPR = D / E;               // pieces per row
  static constexpr int GRP = LPR <= 8 ? 8 : (LPR <= 16 ? 16 : 32);
  static constexpr int RPW = 64 / GRP;            // rows per wave per step
  static constexpr int U = 4;                     // steps per trip (loads in flight per lane: 2U)
  static constexpr int NG = (DEC_THREADS / 64) * RPW;  // lane groups per workgroup
};

// rotated piece `seg` of a head vector x (global), rotate-half convention;
// inv[i] = theta^(-2i/d) (LDS)
template <typename T, int D>
__device__ __forceinline__ void load_rotated_piece(const T* x, int seg, bool rotate, double ps,
                                                   const double* inv, float* out) {
  constexpr int E = Piece<T>::E;
  constexpr int LPR = D / E;
  Piece<T>::unpack(ld16(x + seg * E), out);
  if (!rotate) return;
  const bool first = seg < LPR / 2;
  const int pseg = first ? seg + LPR / 2 : seg - LPR / 2;
  float partner[E];
  Piece<T>::unpack(ld16(x + pseg * E), partner);
  const double two_pi = 6.283185307179586476925286766559;
  const double inv_two_pi = 0.15915494309189533576888376337251;
  const int i0 = (first ? seg : pseg) * E;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    double ang = ps * inv[i0 + e];
    ang -= two_pi * rint(ang * inv_two_pi);
    float sn, cs;
    sincosf((float)ang, &sn, &cs);
    out[e] = first ? out[e] * cs - partner[e] * sn : out[e] * cs + partner[e] * sn;
  }
}

// 0: ordinary append step; 1: <CL> step; 2: token outside [0, L_meta);
// 3: no room for the new row
__device__ __forceinline__ int step_kind(const int32_t* cur_tok, const int32_t* vu,
                                         const int32_t* kv_len, int s, int L_meta, int L_cap) {
  const int t = cur_tok[s];
  if (t < 0 || t >= L_meta) return 2;
  if (vu[(int64_t)s * L_meta + t] == t) return 1;
  const int n = kv_len[s];
  if (n < 0 || n >= L_cap) return 3;
  return 0;
}

template <typename T, int D>
__global__ __launch_bounds__(DEC_THREADS) void decode_chunk_kernel(
    const T* __restrict__ q, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ k_cache, T* __restrict__ v_cache, const int32_t* __restrict__ kv_len,
    const int32_t* __restrict__ cur_tok, const int32_t* __restrict__ vu,
    const int32_t* __restrict__ pos, int32_t L_meta, int32_t H, int32_t L_cap, float qscale,
    int rotate, RopeTab tab, float* __restrict__ part, int32_t n_chunk_max, int32_t n_work) {
  using C = DecCfg<T, D>;
  constexpr int E = C::E, LPR = C::LPR, GRP = C::GRP, RPW = C::RPW, U = C::U, NG = C::NG;
  // chunk-major order: every slice's first chunk is dispatched before any
  // slice's second chunk, so the workgroups that start past a slice's last
  // row (and exit at once) are dispatched last
  const int n_bh = n_work / n_chunk_max;
  const int chunk = blockIdx.x / n_bh;
  const int bh = blockIdx.x % n_bh;
  const int s = bh / H;
  if (step_kind(cur_tok, vu, kv_len, s, L_meta, L_cap) != 0) return;  // combine handles it
  const int n = kv_len[s];
  const int rows = n + 1;
  const int r0 = chunk * DEC_CH;
  if (r0 >= rows) return;
  const int r1 = min(r0 + DEC_CH, rows);
  const int rc = min(r1, n);  // cache rows of this chunk: [r0, rc)

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int g = lane / GRP;      // row slot within the wave
  const int seg = lane % GRP;    // piece within the row
  const bool active = seg < LPR;

  const T* kb = k_cache + (int64_t)bh * L_cap * D;
  const T* vb = v_cache + (int64_t)bh * L_cap * D;
  constexpr int TRIP = (DEC_THREADS / 64) * U * RPW;  // rows per trip of the workgroup
  const int base0 = r0 + wave * U * RPW;

  // streamed rows: the 2U loads of one trip are issued together
  u32x4 kw[U], vw[U];
  auto issue = [&](int base, u32x4* kd, u32x4* vd) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int row = base + u * RPW + g;
      if (row < rc && active) {
        kd[u] = ld16(kb + (int64_t)row * D + seg * E);
        vd[u] = ld16(vb + (int64_t)row * D + seg * E);
      } else {
        kd[u] = u32x4{0, 0, 0, 0};
        vd[u] = u32x4{0, 0, 0, 0};
      }
    }
  };
  __shared__ double inv[D / 2];
  if (rotate && tid < D / 2) inv[tid] = tab.w[tid];
  __syncthreads();

  const double ps = rotate ? (double)pos[(int64_t)s * L_meta + cur_tok[s]] : 0.0;
  float qf[E];
#pragma unroll
  for (int e = 0; e < E; ++e) qf[e] = 0.f;
  if (active) {
    load_rotated_piece<T, D>(q + (int64_t)bh * D, seg, rotate, ps, inv, qf);
#pragma unroll
    for (int e = 0; e < E; ++e) qf[e] *= qscale;  // scores come out in log2 units
  }

  float m = -INFINITY, l = 0.f, acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;

  issue(base0, kw, vw);
  for (int base = base0; base < rc; base += TRIP) {
    float sc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[E];
      Piece<T>::unpack(kw[u], kf);
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) d = fmaf(qf[e], kf[e], d);
      d = group_sum<GRP>(d);
      sc[u] = (base + u * RPW + g < rc) ? d : -INFINITY;
    }
    float mx = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mx = fmaxf(mx, sc[u]);
    if (mx != -INFINITY) {
      const float alpha = exp2f(m - mx);  // m == -inf gives 0
      l *= alpha;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2f(sc[u] - mx);
        l += p;
        float vf[E];
        Piece<T>::unpack(vw[u], vf);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(p, vf[e], acc[e]);
      }
      m = mx;
    }
    if (base + TRIP < rc) issue(base + TRIP, kw, vw);
  }

  // the new row: rotated k_new, v_new; written to the cache by this chunk
  if (n >= r0 && n < r1 && wave == 0 && g == 0) {
    float kf[E], vf[E];
#pragma unroll
    for (int e = 0; e < E; ++e) { kf[e] = 0.f; vf[e] = 0.f; }
    if (active) {
      load_rotated_piece<T, D>(k_new + (int64_t)bh * D, seg, rotate, ps, inv, kf);
      // score with the stored (rounded) key, exactly as later steps will see it
      Piece<T>::unpack(Piece<T>::pack(kf), kf);
      Piece<T>::unpack(ld16(v_new + (int64_t)bh * D + seg * E), vf);
    }
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) d = fmaf(qf[e], kf[e], d);
    d = group_sum<GRP>(d);
    const float mx = fmaxf(m, d);
    const float alpha = exp2f(m - mx);
    const float p = exp2f(d - mx);
    l = l * alpha + p;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = fmaf(p, vf[e], acc[e] * alpha);
    m = mx;
    if (active) {
      st16(k_cache + ((int64_t)bh * L_cap + n) * D + seg * E, Piece<T>::pack(kf));
      st16(v_cache + ((int64_t)bh * L_cap + n) * D + seg * E,
           ld16(v_new + (int64_t)bh * D + seg * E));
    }
  }

  // merge the lane groups of the workgroup into this chunk's partial
  __shared__ float sm[NG], sl[NG];
  __shared__ float sacc[NG][D];
  const int grp = wave * RPW + g;
  if (active) {
#pragma unroll
    for (int e = 0; e < E; ++e) sacc[grp][seg * E + e] = acc[e];
    if (seg == 0) { sm[grp] = m; sl[grp] = l; }
  }
  __syncthreads();
  float* out = part + ((int64_t)bh * n_chunk_max + chunk) * (D + 2);
  if (tid < D) {
    float M = -INFINITY;
    for (int i = 0; i < NG; ++i) M = fmaxf(M, sm[i]);
    float Lsum = 0.f, ov = 0.f;
    for (int i = 0; i < NG; ++i) {
      if (sm[i] == -INFINITY) continue;
      const float w = exp2f(sm[i] - M);
      Lsum += sl[i] * w;
      ov += sacc[i][tid] * w;
    }
    out[2 + tid] = ov;
    if (tid == 0) { out[0] = M; out[1] = Lsum; }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(128) void decode_combine_kernel(
    const T* __restrict__ v_new, const int32_t* __restrict__ kv_len,
    const int32_t* __restrict__ cur_tok, const int32_t* __restrict__ vu, int32_t L_meta,
    int32_t H, int32_t L_cap, const float* __restrict__ part, int32_t n_chunk_max,
    T* __restrict__ o, int32_t* __restrict__ status) {
  constexpr int E = Piece<T>::E;
  const int bh = blockIdx.x;
  const int s = bh / H;
  const int tid = threadIdx.x;
  const int kind = step_kind(cur_tok, vu, kv_len, s, L_meta, L_cap);
  if (kind >= 2 && tid == 0 && (bh % H) == 0 && status)
    atomicOr(status, kind == 2 ? SCKV_STATUS_TOKEN : SCKV_STATUS_CAP);
  __shared__ float res[D];
  __shared__ float cw[128];  // chunk weights exp2(m_c - M), a block of 128 chunks at a time
  __shared__ float red[2];
  if (kind != 0) {
    if (tid < D) {
      float r = NAN;
      if (kind == 1) {
        const T* vn = v_new + (int64_t)bh * D;
        if constexpr (sizeof(T) == 2) r = bf16_lo((uint32_t)vn[tid]);
        else r = vn[tid];
      }
      res[tid] = r;
    }
  } else {
    const int nch = (kv_len[s] + 1 + DEC_CH - 1) / DEC_CH;
    const float* p = part + (int64_t)bh * n_chunk_max * (D + 2);
    // global max over the chunk maxima (one wave)
    if (tid < 64) {
      float M = -INFINITY;
      for (int c = tid; c < nch; c += 64) M = fmaxf(M, p[c * (D + 2)]);
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
      if (tid == 0) red[0] = M;
    }
    __syncthreads();
    const float M = red[0];
    float Lsum = 0.f, acc = 0.f;
    for (int c0 = 0; c0 < nch; c0 += 128) {
      const int c = c0 + tid;
      if (c < nch) {
        const float mc = p[c * (D + 2)];
        const float w = (mc == -INFINITY) ? 0.f : exp2f(mc - M);
        cw[tid] = w;
      }
      __syncthreads();
      const int cn = min(128, nch - c0);
      if (tid < D) {
#pragma unroll 8
        for (int i = 0; i < cn; ++i) {
          const float w = cw[i];
          const float* pc = p + (c0 + i) * (D + 2);
          Lsum = fmaf(pc[1], w, Lsum);
          acc = fmaf(pc[2 + tid], w, acc);
        }
      }
      __syncthreads();
    }
    if (tid < D) res[tid] = acc / Lsum;
  }
  __syncthreads();
  if (tid < D / E) {
    float f[E];
#pragma unroll
    for (int e = 0; e < E; ++e) f[e] = res[tid * E + e];
    st16(o + (int64_t)bh * D + tid * E, Piece<T>::pack(f));
  }
}

static int n_chunks(int L_cap) { return (L_cap + DEC_CH - 1) / DEC_CH; }

template <typename T, int D>
static int launch_decode(const void* q, const void* k_new, const void* v_new, void* k_cache,
                         void* v_cache, const int32_t* kv_len, const int32_t* cur_tok,
                         const int32_t* vu, const int32_t* pos, int32_t L_meta, void* o,
                         int32_t b, int32_t H, int32_t L_cap, float scale, float theta,
                         void* ws, int32_t* status, hipStream_t stream) {
  RopeTab tab;
  for (int i = 0; i < 40; ++i) tab.w[i] = 0.0;
  const int rotate = theta > 0.f ? 1 : 0;
  if (rotate)
    for (int i = 0; i < D / 2; ++i) tab.w[i] = std::pow((double)theta, -2.0 * i / D);
  const int nc = n_chunks(L_cap);
  float* part = static_cast<float*>(ws);
  const int n_work = b * H * nc;
  decode_chunk_kernel<T, D><<<n_work, DEC_THREADS, 0, stream>>>(
      static_cast<const T*>(q), static_cast<const T*>(k_new), static_cast<const T*>(v_new),
      static_cast<T*>(k_cache), static_cast<T*>(v_cache), kv_len, cur_tok, vu, pos, L_meta, H,
      L_cap, scale * LOG2E, rotate, tab, part, nc, n_work);
  int rc = hip_check(hipGetLastError(), "compacted_decode_attn: chunk launch");
  if (rc) return rc;
  decode_combine_kernel<T, D><<<b * H, 128, 0, stream>>>(
      static_cast<const T*>(v_new), kv_len, cur_tok, vu, L_meta, H, L_cap, part, nc,
      static_cast<T*>(o), status);
  return hip_check(hipGetLastError(), "compacted_decode_attn: combine launch");
}

}  // namespace sckv

using namespace sckv;

extern "C" size_t sckv_decode_workspace_bytes(int32_t b, int32_t H, int32_t L_cap, int32_t d_head) {
  if (b <= 0 || H <= 0 || L_cap <= 0 || d_head <= 0) return 0;
  return (size_t)b * H * n_chunks(L_cap) * (d_head + 2) * sizeof(float);
}

extern "C" int compacted_decode_attn(const void* q, const void* k_new, const void* v_new,
                                     void* k_cache, void* v_cache, const int32_t* kv_len,
                                     const int32_t* cur_tok, const int32_t* vu,
                                     const int32_t* pos, int32_t L_meta, void* o, int32_t b,
                                     int32_t H, int32_t L_cap, int32_t d_head, sckv_dtype dt,
                                     float scale, float rope_theta, void* ws, size_t ws_bytes,
                                     int32_t* status, hipStream_t stream) {
  clear_error();
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !kv_len || !cur_tok || !vu || !o || !ws)
    return fail(SCKV_EINVAL, "compacted_decode_attn: null pointer");
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, "compacted_decode_attn: unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, "compacted_decode_attn: d_head must be 64 or 80");
  if (b <= 0 || H <= 0 || L_cap <= 0 || L_meta <= 0)
    return fail(SCKV_EINVAL, "compacted_decode_attn: sizes must be positive");
  if ((int64_t)b * H * n_chunks(L_cap) > 0x7fffffff)
    return fail(SCKV_EUNSUP, "compacted_decode_attn: b*H*chunks too large");
  if (!(scale > 0.f) || std::isinf(scale)) return fail(SCKV_EINVAL, "compacted_decode_attn: scale must be finite and > 0");
  if (!(rope_theta >= 0.f) || std::isinf(rope_theta))
    return fail(SCKV_EINVAL, "compacted_decode_attn: rope_theta must be finite and >= 0");
  if (rope_theta > 0.f && !pos) return fail(SCKV_EINVAL, "compacted_decode_attn: null pos");
  if (ws_bytes < sckv_decode_workspace_bytes(b, H, L_cap, d_head))
    return fail(SCKV_EINVAL, "compacted_decode_attn: workspace too small");
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
      !aligned16(v_cache) || !aligned16(o) || !aligned16(ws))
    return fail(SCKV_EINVAL, "compacted_decode_attn: buffers must be 16-byte aligned");
  const int32_t* p = pos ? pos : vu;  // pos is read only when rotating
  if (dt == SCKV_BF16)
    return d_head == 64
               ? launch_decode<uint16_t, 64>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream)
               : launch_decode<uint16_t, 80>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream);
  return d_head == 64
             ? launch_decode<float, 64>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream)
             : launch_decode<float, 80>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream);
}
