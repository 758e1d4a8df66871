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
#include <mutex>
#include <string>

#include "sckv_common.h"

namespace sckv {

// Launch shapes, measured on MI355X over three decode shapes: 2048 slices of
// about 560 rows (d=64), 512 slices of about 2100 rows (d=80, rotary) and
// 8192 slices of about 1200 rows (d=80, rotary).  A slice is one (sequence,
// head) pair.
//  * Fewer than DEC_SINGLE_MIN slices: each slice is cut into chunks of
//    about DEC_CH rows, one 4-wave workgroup each, and a second kernel merges
//    the chunk partials.
//  * Otherwise one workgroup per slice writes the output itself (no second
//    launch).  fp32: 512 threads below DEC_NARROW_MIN slices, 256 from there
//    on.  bf16: the most waves per slice (4, 2 or 1; 1 only where d <= 64)
//    with which every wave of the launch is resident at once (the kernel
//    holds two waves per SIMD), so the launch runs in one round; where even
//    one wave per slice exceeds that, 4 waves, whose shorter workgroups
//    balance the rounds best.  Measured: 512 slices (d=80) 4 waves; 2048
//    slices (d=64) 1 wave 2% faster than 2 and 4% faster than 4; 8192
//    slices (d=80) 4 waves 2.5% faster than 2.
constexpr int DEC_CH = 1024;
constexpr int DEC_SINGLE_MIN = 512;
constexpr int DEC_NARROW_MIN = 1024;
constexpr int DEC_WAVES_PER_SIMD = 2;  // decode_mfma_kernel's occupancy (its register count)
constexpr int DEC_SPEC2_ROWS = 512;    // cache rows per wave from which two blocks are speculated

// compute units of the current device, asked once per device
static int device_cus(int* cus) {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  int rc = hip_check(hipGetDevice(&dev), "compacted_decode_attn: hipGetDevice");
  if (rc) return rc;
  if (dev < 0 || dev >= 64) return fail(SCKV_EUNSUP, "compacted_decode_attn: device index above 63");
  std::lock_guard<std::mutex> lock(mu);
  if (cached[dev] == 0) {
    int n = 0;
    rc = hip_check(hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev),
                   "compacted_decode_attn: hipDeviceGetAttribute");
    if (rc) return rc;
    cached[dev] = n > 0 ? n : 1;
  }
  *cus = cached[dev];
  return 0;
}
constexpr int DEC_THREADS = 256;  // fp32 split chunks
constexpr float LOG2E = 1.4426950408889634f;

struct RopeTab {
  double w[40];  // theta^(-2i/d), i < d/2
};

template <typename T, int D, int THREADS>
struct DecCfg {
  static constexpr int E = Piece<T>::E;           // elements per piece
  static constexpr int LPR = D / E;               // pieces per row
  static constexpr int GRP = LPR <= 8 ? 8 : (LPR <= 16 ? 16 : 32);
  static constexpr int RPW = 64 / GRP;            // rows per wave per step
  static constexpr int U = 4;                     // steps per trip (loads in flight per lane: 2U)
  static constexpr int NG = (THREADS / 64) * RPW;  // lane groups per workgroup
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

// Writes the final output of a slice whose step is not an ordinary append
// (kind 1: <CL>, the output is v_new; kind 2/3: failure, NaN and a status
// bit).  `tid` runs over `nthr` threads.
// A slice's rows split into n chunks of `rows` rows (the last one shorter)
// of at most about `ch` rows each.  Chunk starts are multiples of 16 rows:
// a wave then reads whole 128-byte lines (a bf16 row of 80 elements is 160
// bytes, so only every fourth row starts on a line; a chunk that started
// between would make every load of its wave span one line more).
struct ChunkPlan {
  int n, rows;
};
constexpr int DEC_ALIGN = 16;
// rows and ch are positive ints, so every sum below fits in 32 unsigned bits
__device__ __forceinline__ ChunkPlan chunk_plan(int rows, int ch) {
  const uint32_t r = (uint32_t)rows, c = (uint32_t)ch;
  const uint32_t n0 = (r + c - 1) / c;
  const uint32_t per = (r + n0 - 1) / n0;
  const uint32_t cr = (per + DEC_ALIGN - 1) / DEC_ALIGN * DEC_ALIGN;
  ChunkPlan p;
  p.rows = (int)cr;
  p.n = (int)((r + cr - 1) / cr);  // <= n0
  return p;
}

template <typename T, int D>
__device__ __forceinline__ void write_special(int kind, const T* v_new, T* o, int32_t* status,
                                              int bh, int H, int tid, int nthr) {
  if (kind >= 2 && tid == 0 && (bh % H) == 0 && status)
    atomicOr(status, kind == 2 ? SCKV_STATUS_TOKEN : SCKV_STATUS_CAP);
  for (int i = tid; i < D; i += nthr) {
    if (kind == 1) o[(int64_t)bh * D + i] = v_new[(int64_t)bh * D + i];
    else if constexpr (sizeof(T) == 2) o[(int64_t)bh * D + i] = (T)0x7fc0;  // bf16 NaN
    else o[(int64_t)bh * D + i] = NAN;
  }
}

// FINAL: the workgroup covers the whole slice (one chunk of L_cap rows) and
// writes the output itself; otherwise it writes a partial for the combine.
template <typename T, int D, int THREADS, bool FINAL>
__global__ __launch_bounds__(THREADS) void decode_chunk_kernel(
    const T* __restrict__ q, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ k_cache, T* __restrict__ v_cache, const int32_t* __restrict__ kv_len,
    const int32_t* __restrict__ cur_tok, const int32_t* __restrict__ vu,
    const int32_t* __restrict__ pos, int32_t L_meta, int32_t H, int32_t L_cap, float qscale,
    int rotate, RopeTab tab, float* __restrict__ part, int32_t n_chunk_max, int32_t n_work,
    int32_t ch, T* __restrict__ o, int32_t* __restrict__ status) {
  using C = DecCfg<T, D, THREADS>;
  constexpr int E = C::E, LPR = C::LPR, GRP = C::GRP, RPW = C::RPW, U = C::U, NG = C::NG;
  // chunk-major order: every slice's first chunk is dispatched before any
  // slice's second chunk, so the workgroups that start past a slice's last
  // row (and exit at once) are dispatched last
  const int n_bh = n_work / n_chunk_max;
  const int chunk = blockIdx.x / n_bh;
  const int bh = blockIdx.x % n_bh;
  const int s = bh / H;
  const int kind = step_kind(cur_tok, vu, kv_len, s, L_meta, L_cap);
  if (kind != 0) {  // the combine handles it, or this workgroup when FINAL
    if constexpr (FINAL) write_special<T, D>(kind, v_new, o, status, bh, H, threadIdx.x, THREADS);
    return;
  }
  const int n = kv_len[s];
  const int rows = n + 1;  // cache rows and the new row
  const ChunkPlan cp = chunk_plan(rows, ch);
  if (chunk >= cp.n) return;
  const int r0 = chunk * cp.rows;
  const int r1 = min(r0 + cp.rows, rows);
  const int rc = min(r1, n);  // cache rows of this chunk: [r0, rc)

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int g = lane / GRP;      // row slot within the wave
  const int seg = lane % GRP;    // piece within the row
  const bool active = seg < LPR;

  const T* kb = k_cache + (int64_t)bh * L_cap * D;
  const T* vb = v_cache + (int64_t)bh * L_cap * D;
  constexpr int TRIP = (THREADS / 64) * U * RPW;  // rows per trip of the workgroup
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
  __shared__ float res[D];
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
    if constexpr (FINAL) {
      res[tid] = ov / Lsum;
    } else {
      float* out = part + ((int64_t)bh * n_chunk_max + chunk) * (D + 2);
      out[2 + tid] = ov;
      if (tid == 0) { out[0] = M; out[1] = Lsum; }
    }
  }
  if constexpr (FINAL) {
    __syncthreads();
    if (tid < D / E) {
      float f[E];
#pragma unroll
      for (int e = 0; e < E; ++e) f[e] = res[tid * E + e];
      st16(o + (int64_t)bh * D + tid * E, Piece<T>::pack(f));
    }
  }
}

// One wave per slice: log-sum-exp merge of the slice's chunk partials, 64
// chunks at a time (lane c holds chunk c's weight; the output elements are
// spread over the lanes).
template <typename T, int D>
__global__ __launch_bounds__(64) void decode_combine_kernel(
    const T* __restrict__ v_new, const int32_t* __restrict__ kv_len,
    const int32_t* __restrict__ cur_tok, const int32_t* __restrict__ vu, int32_t L_meta,
    int32_t H, int32_t L_cap, const float* __restrict__ part, int32_t n_chunk_max, int32_t ch,
    T* __restrict__ o, int32_t* __restrict__ status, int32_t ring) {
  const int bh = blockIdx.x;
  const int s = bh / H;
  const int lane = threadIdx.x;
  int kind;
  if (ring > 0) {  // the ring is always full: only token range and <CL> steps
    const int t = cur_tok[s];
    kind = (t < 0 || t >= L_meta) ? 2 : (vu[(int64_t)s * L_meta + t] == t ? 1 : 0);
  } else {
    kind = step_kind(cur_tok, vu, kv_len, s, L_meta, L_cap);
  }
  if (kind != 0) {
    write_special<T, D>(kind, v_new, o, status, bh, H, lane, 64);
    return;
  }
  const int nch = chunk_plan((ring > 0 ? ring : kv_len[s]) + 1, ch).n;
  const float* p = part + (int64_t)bh * n_chunk_max * (D + 2);
  constexpr int PER = (D + 63) / 64;  // output elements per lane
  float M = -INFINITY, lsum = 0.f, acc[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] = 0.f;
  for (int c0 = 0; c0 < nch; c0 += 64) {
    const int c = c0 + lane;
    float mc = -INFINITY, lc = 0.f;
    if (c < nch) {
      mc = p[c * (D + 2)];
      lc = p[c * (D + 2) + 1];
    }
    float mb = mc;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mb = fmaxf(mb, __shfl_xor(mb, off, 64));
    const float mn = fmaxf(M, mb);    // finite: every chunk holds a row
    const float sc = exp2f(M - mn);   // 0 on the first block (M = -inf)
    lsum *= sc;
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] *= sc;
    const float w = c < nch ? exp2f(mc - mn) : 0.f;
    lsum = fmaf(lc, w, lsum);
    const int cn = min(64, nch - c0);
#pragma unroll 4
    for (int i = 0; i < cn; ++i) {
      const float wi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), i));
      const float* pc = p + (c0 + i) * (D + 2) + 2;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (lane + 64 * j < D) acc[j] = fmaf(pc[lane + 64 * j], wi, acc[j]);
    }
    M = mn;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lsum += __shfl_xor(lsum, off, 64);
  const float inv = 1.f / lsum;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = lane + 64 * j;
    if (e < D) {
      if constexpr (sizeof(T) == 2) o[(int64_t)bh * D + e] = f32_to_bf16(acc[j] * inv);
      else o[(int64_t)bh * D + e] = acc[j] * inv;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 caches: scores on the matrix cores
// ---------------------------------------------------------------------------
// A wave takes 32-row blocks of the chunk (block i of the chunk goes to wave
// i mod NW).  Lane l owns key row l%32 of the block and elements
// 16kk + 8(l/32) .. +7 (kk < D/16) of that row's key and value: exactly the
// B operand of v_mfma_f32_32x32x16_bf16 for B[k][n] = K[n][k].  With the A
// operand holding q in every one of its 32 rows, every column n of the
// result is the score of key n, so each lane ends up with the score of its
// own key and weighs its own value elements with it (no cross-lane traffic
// per row).  q is split into two bf16 terms (hi + lo) so that the scores
// keep about fp32 accuracy.  The running maximum is raised only when a block
// maximum exceeds it by DM_RESCALE (log2 units), which keeps rescaling rare;
// accumulated weights stay below 2^DM_RESCALE per row.  The next block's
// rows are in flight while a block is computed.
constexpr float DM_RESCALE = 8.f;

// Sums v[0..NV) over the 32 lanes of each half-wave.  While NV is even a
// step halves the values a lane keeps (the lane whose MASK bit is set keeps
// the upper half); odd counts finish with plain butterflies.  On return the
// lane holds the sums of values [base, base + count).
template <int NV, int MASK>
__device__ __forceinline__ void half_wave_reduce(float* v, int lane, int& base) {
  if constexpr (MASK > 0) {
    if constexpr (NV % 2 == 0) {
      constexpr int HV = NV / 2;
      const bool up = (lane & MASK) != 0;
#pragma unroll
      for (int j = 0; j < HV; ++j) {
        const float send = up ? v[j] : v[j + HV];
        const float keep = up ? v[j + HV] : v[j];
        v[j] = keep + __shfl_xor(send, MASK, 64);
      }
      if (up) base += HV;
      half_wave_reduce<HV, MASK / 2>(v, lane, base);
    } else {
#pragma unroll
      for (int j = 0; j < NV; ++j) v[j] += __shfl_xor(v[j], MASK, 64);
      half_wave_reduce<NV, MASK / 2>(v, lane, base);
    }
  }
}
template <int NV, int MASK>
constexpr int half_wave_count() {
  if constexpr (MASK == 0) return NV;
  else if constexpr (NV % 2 == 0) return half_wave_count<NV / 2, MASK / 2>();
  else return half_wave_count<NV, MASK / 2>();
}

template <int D, int NW, bool FINAL, bool SPEC2 = false>
__global__ __launch_bounds__(NW * 64) void decode_mfma_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, uint16_t* __restrict__ k_cache,
    uint16_t* __restrict__ v_cache, const int32_t* __restrict__ kv_len,
    const int32_t* __restrict__ cur_tok, const int32_t* __restrict__ vu,
    const int32_t* __restrict__ pos, int32_t L_meta, int32_t H, int32_t L_cap, float qscale,
    int rotate, RopeTab tab, float* __restrict__ part, int32_t n_chunk_max, int32_t n_work,
    int32_t ch, uint16_t* __restrict__ o, int32_t* __restrict__ status, int32_t ring) {
  constexpr int KS = D / 16;     // k steps of 16 elements
  constexpr int NA = 8 * KS;     // value elements per lane
  constexpr int THREADS = NW * 64;
  constexpr int HD = D / 2;
  // new-row elements: one per thread of the workgroup, then one or two per
  // lane of wave 0 for the score
  static_assert(D >= 64 && D <= 128 && D % 16 == 0 && D <= NW * 64, "head size");
  // chunk-major order (as in decode_chunk_kernel); a one-chunk launch has
  // one workgroup per slice
  const int n_bh = FINAL ? n_work : n_work / n_chunk_max;
  const int chunk = FINAL ? 0 : (int)blockIdx.x / n_bh;
  const int bh = FINAL ? (int)blockIdx.x : (int)blockIdx.x % n_bh;
  const int s = bh / H;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int kr = lane & 31;
  const int h = lane >> 5;

  // Everything the setup reads is wave-uniform and goes through scalar
  // loads, whose counter is separate from that of the vector loads: the
  // first two blocks of key/value rows are issued as soon as the slice
  // length is known and arrive while q is prepared.  The block addresses use
  // the length clamped into the cache, so they are valid whatever the step
  // turns out to be.
  // ring > 0 (local-attention comparator): rows [0, ring) are a ring of the
  // ring most recent tokens, token t at row t mod ring; the new token
  // replaces the oldest, whose row is not attended
  const int n_raw = ring > 0 ? ring : kv_len[s];
  const int t_raw = cur_tok[s];
  // the new row: thread tid < D takes element tid of k_new and v_new and
  // the element k_new rotates against.  These vector loads go out before the
  // block loads (the counter retires in issue order), so the new row is
  // ready before the first block and its latency hides under the stream.
  // Threads past D re-read element D - 1.
  const int te = min(tid, D - 1);
  const int tp = te < HD ? te + HD : te - HD;
  const uint16_t kx_raw = k_new[(int64_t)bh * D + te];
  const uint16_t kp_raw = k_new[(int64_t)bh * D + tp];
  const uint16_t vx_raw = v_new[(int64_t)bh * D + te];
  // A one-chunk launch (FINAL) starts its slice at row 0, so its first block
  // is rows 32*wave.. whatever the slice length: it is issued before the
  // length arrives (rows past the slice's end are neutralised below).
  const uint16_t* kb = k_cache + (int64_t)bh * L_cap * D;
  const uint16_t* vb = v_cache + (int64_t)bh * L_cap * D;
  auto load_row = [&](int row, u32x4* kd, u32x4* vd) {
    const uint16_t* kp = kb + (int64_t)row * D + 8 * h;
    const uint16_t* vp = vb + (int64_t)row * D + 8 * h;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) kd[kk] = ld16(kp + 16 * kk);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) vd[kk] = ld16(vp + 16 * kk);
  };
  u32x4 kA[KS], vA[KS], kB[KS], vB[KS];
  if constexpr (FINAL) load_row(min(32 * wave + kr, L_cap - 1), kA, vA);
  // with SPEC2 (chosen by the host for caches large enough that slices are
  // taken to be long) the second block is issued before the length too
  if constexpr (FINAL && SPEC2) load_row(min(32 * (wave + NW) + kr, L_cap - 1), kB, vB);
  const uint32_t* qw = reinterpret_cast<const uint32_t*>(q + (int64_t)bh * D);
  uint32_t qword[HD];
#pragma unroll
  for (int j = 0; j < HD; ++j) qword[j] = qw[j];
  const bool t_ok = t_raw >= 0 && t_raw < L_meta;
  const int vu_t = t_ok ? vu[(int64_t)s * L_meta + t_raw] : 0;
  const int pos_t = (rotate && t_ok) ? pos[(int64_t)s * L_meta + t_raw] : 0;

  const int n = ring > 0 ? ring : min(max(n_raw, 0), L_cap - 1);
  const int slot = (ring > 0 && t_ok) ? t_raw % ring : -1;  // row of the new token (ring)
  const int rows = n + 1;
  const ChunkPlan cp = chunk_plan(rows, ch);
  const int r0 = chunk * cp.rows;
  const int r1 = min(r0 + cp.rows, rows);
  const int rc = min(r1, n);  // cache rows of this chunk: [r0, rc)
  const int nblk = chunk < cp.n ? (rc - r0 + 31) / 32 : 0;
  const bool holds_new = n >= r0 && n < r1;

  // rows past rc re-read row rc-1 (row 0 where the chunk has no rows);
  // their scores are masked
  auto load_blk = [&](int i, u32x4* kd, u32x4* vd) {
    load_row(max(min(r0 + 32 * i + kr, rc - 1), 0), kd, vd);
  };
  // issued whether or not the wave has these blocks, so that the counter
  // waits below stay exact on every path
  if constexpr (FINAL) {
    if constexpr (!SPEC2) load_blk(wave + NW, kB, vB);
    // a short slice: rows past its end were read too.  Their scores are
    // masked; their values are zeroed so that whatever those rows hold
    // (they may never have been written) adds exactly nothing.
    if (32 * wave + 32 > rc) {
      const bool a_in = 32 * wave + kr < rc;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) vA[kk] = a_in ? vA[kk] : u32x4{0, 0, 0, 0};
    }
    if constexpr (SPEC2) {
      if (32 * (wave + NW) + 32 > rc) {
        const bool b_in = 32 * (wave + NW) + kr < rc;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) vB[kk] = b_in ? vB[kk] : u32x4{0, 0, 0, 0};
      }
    }
  } else {
    load_blk(wave, kA, vA);
    load_blk(wave + NW, kB, vB);
  }

  // the step kind, with the precedence of step_kind()
  const int kind = !t_ok ? 2
                   : (vu_t == t_raw ? 1 : ((ring == 0 && (n_raw < 0 || n_raw >= L_cap)) ? 3 : 0));
  if (kind != 0) {
    if constexpr (FINAL) write_special<uint16_t, D>(kind, v_new, o, status, bh, H, tid, THREADS);
    return;
  }
  if (chunk >= cp.n) return;

  // rotated q and k elements tid (tid < D), q from the words held in scalar
  // registers; both turn by the same angle.  The key is rounded to bf16 as
  // stored; its product with q and the value element go to LDS.
  __shared__ float qs[D], kqs[D], vs[D];
  if (tid < D) {
    uint32_t xw = 0, pw = 0;
#pragma unroll
    for (int j = 0; j < HD; ++j) {
      xw = (tid >> 1) == j ? qword[j] : xw;
      pw = (tp >> 1) == j ? qword[j] : pw;
    }
    float x = (tid & 1) ? bf16_hi(xw) : bf16_lo(xw);
    float kx = bf16_lo((uint32_t)kx_raw);
    if (rotate) {
      const float pv = (tp & 1) ? bf16_hi(pw) : bf16_lo(pw);
      const float kp = bf16_lo((uint32_t)kp_raw);
      double w = 0.0;
#pragma unroll
      for (int j = 0; j < HD; ++j) w = (tid % HD) == j ? tab.w[j] : w;
      const double two_pi = 6.283185307179586476925286766559;
      const double inv_two_pi = 0.15915494309189533576888376337251;
      double ang = (double)pos_t * w;
      ang -= two_pi * rint(ang * inv_two_pi);
      float sn, cs;
      sincosf((float)ang, &sn, &cs);
      x = tid < HD ? x * cs - pv * sn : x * cs + pv * sn;
      kx = tid < HD ? kx * cs - kp * sn : kx * cs + kp * sn;
    }
    const uint16_t kq = f32_to_bf16(kx);
    qs[tid] = x;
    kqs[tid] = x * bf16_lo((uint32_t)kq);
    vs[tid] = bf16_lo((uint32_t)vx_raw);
    if (holds_new) {
      const int64_t dst = (int64_t)bh * L_cap + (ring > 0 ? slot : n);
      k_cache[dst * D + tid] = kq;
      v_cache[dst * D + tid] = vx_raw;
    }
  }
  __syncthreads();

  bf16x8 qhi[KS], qlo[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4 wh, wl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float x0 = qs[16 * kk + 8 * h + 2 * i], x1 = qs[16 * kk + 8 * h + 2 * i + 1];
      const uint32_t hw = pack_bf16x2(x0, x1);
      wh[i] = hw;
      wl[i] = pack_bf16x2(x0 - bf16_lo(hw), x1 - bf16_hi(hw));
    }
    qhi[kk] = __builtin_bit_cast(bf16x8, wh);
    qlo[kk] = __builtin_bit_cast(bf16x8, wl);
  }

  float M = -INFINITY, l = 0.f, acc[NA];
#pragma unroll
  for (int a = 0; a < NA; ++a) acc[a] = 0.f;
  // takes a score (wave-uniform block maximum over lanes); returns its weight
  auto weigh = [&](float sc) {
    float mb = sc;
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) mb = fmaxf(mb, __shfl_xor(mb, off, 64));
    if (mb > M + DM_RESCALE) {
      const float f = exp2f(M - mb);  // 0 while M = -inf
      l *= f;
#pragma unroll
      for (int a = 0; a < NA; ++a) acc[a] *= f;
      M = mb;
    }
    return exp2f(sc - M);
  };
  auto compute = [&](int i, const u32x4* kd, const u32x4* vd) {
    f32x16 c;
#pragma unroll
    for (int v = 0; v < 16; ++v) c[v] = 0.f;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const bf16x8 kv = __builtin_bit_cast(bf16x8, kd[kk]);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qhi[kk], kv, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qlo[kk], kv, c, 0, 0, 0);
    }
    const int row = r0 + 32 * i + kr;
    const float sc = (row < rc && row != slot) ? c[0] * qscale : -INFINITY;
    const float p = weigh(sc);
    if (h == 0) l += p;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t w = vd[kk][j];
        acc[8 * kk + 2 * j] = fmaf(p, bf16_lo(w), acc[8 * kk + 2 * j]);
        acc[8 * kk + 2 * j + 1] = fmaf(p, bf16_hi(w), acc[8 * kk + 2 * j + 1]);
      }
    }
  };

  // the new row opens the state of wave 0: its score is the sum of the
  // products in LDS; lanes 0 and 32 take the value elements they own and
  // lane 0 counts the weight
  if (holds_new && wave == 0) {
    float prod = kqs[lane];
    if (lane + 64 < D) prod += kqs[lane + 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) prod += __shfl_xor(prod, off, 64);
    const float p = weigh(prod * qscale);
    if (lane == 0) l += p;
    if (kr == 0) {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[8 * kk + j] = p * vs[16 * kk + 8 * h + j];
      }
    }
  }

  // blocks wave, wave + NW are in flight; each computed buffer is refilled
  // with the block 2 NW further on.  The steady state loads without a
  // condition, so each buffer is written in place and the loop carries no
  // register copies (a copy would have to wait for its load to land).
  int i = wave;
  for (; i + 3 * NW < nblk; i += 2 * NW) {
    compute(i, kA, vA);
    load_blk(i + 2 * NW, kA, vA);
    compute(i + NW, kB, vB);
    load_blk(i + 3 * NW, kB, vB);
  }
  // at most three blocks remain: i and i + NW in flight, i + 2 NW to load
  if (i < nblk) {
    compute(i, kA, vA);
    if (i + 2 * NW < nblk) load_blk(i + 2 * NW, kA, vA);
  }
  if (i + NW < nblk) compute(i + NW, kB, vB);
  if (i + 2 * NW < nblk) compute(i + 2 * NW, kA, vA);

  // wave partials: l over the wave, values over each half-wave
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) l += __shfl_xor(l, off, 64);
  int base = 0;
  half_wave_reduce<NA, 16>(acc, lane, base);
  constexpr int NF = half_wave_count<NA, 16>();
  __shared__ float sm[NW], sl[NW];
  __shared__ float sacc[NW][D];
#pragma unroll
  for (int j = 0; j < NF; ++j) {
    const int a = base + j;
    sacc[wave][16 * (a / 8) + 8 * h + a % 8] = acc[j];
  }
  if (lane == 0) { sm[wave] = M; sl[wave] = l; }
  __syncthreads();
  __shared__ float res[D];
  if (tid < D) {
    float Mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) Mx = fmaxf(Mx, sm[w]);
    float Ls = 0.f, ov = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (sm[w] == -INFINITY) continue;
      const float f = exp2f(sm[w] - Mx);
      Ls += sl[w] * f;
      ov += sacc[w][tid] * f;
    }
    if constexpr (FINAL) {
      res[tid] = ov / Ls;
    } else {
      float* out = part + ((int64_t)bh * n_chunk_max + chunk) * (D + 2);
      out[2 + tid] = ov;
      if (tid == 0) { out[0] = Mx; out[1] = Ls; }
    }
  }
  if constexpr (FINAL) {
    __syncthreads();
    if (tid < D / 8) {
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = res[tid * 8 + e];
      st16(o + (int64_t)bh * D + tid * 8, Piece<uint16_t>::pack(f));
    }
  }
}

static int n_chunks(int L_cap) { return (L_cap + DEC_CH - 1) / DEC_CH; }

template <typename T, int D>
static int launch_decode(const void* q, const void* k_new, const void* v_new, void* k_cache,
                         void* v_cache, const int32_t* kv_len, const int32_t* cur_tok,
                         const int32_t* vu, const int32_t* pos, int32_t L_meta, void* o,
                         int32_t b, int32_t H, int32_t L_cap, float scale, float theta,
                         void* ws, int32_t* status, hipStream_t stream, int32_t ring = 0) {
  RopeTab tab;
  for (int i = 0; i < 40; ++i) tab.w[i] = 0.0;
  const int rotate = theta > 0.f ? 1 : 0;
  if (rotate)
    for (int i = 0; i < D / 2; ++i) tab.w[i] = std::pow((double)theta, -2.0 * i / D);
  float* part = static_cast<float*>(ws);
  const T* qq = static_cast<const T*>(q);
  const T* kn = static_cast<const T*>(k_new);
  const T* vn = static_cast<const T*>(v_new);
  T* kc = static_cast<T*>(k_cache);
  T* vc = static_cast<T*>(v_cache);
  T* out = static_cast<T*>(o);
  const float qs = scale * LOG2E;
  const int slices = b * H;
  if (slices >= DEC_SINGLE_MIN) {
    const bool narrow = slices >= DEC_NARROW_MIN;
    if constexpr (sizeof(T) == 2) {
      int cus = 0;
      const int rc = device_cus(&cus);
      if (rc) return rc;
      const int64_t slots = (int64_t)cus * 4 * DEC_WAVES_PER_SIMD;  // resident waves
      const int nw = (int64_t)slices * 4 <= slots   ? 4
                     : (int64_t)slices * 2 <= slots ? 2
                     : slices <= slots              ? (D <= 64 ? 1 : 2)
                                                    : 4;
      // A cache of at least DEC_SPEC2_ROWS rows per wave of a slice is taken
      // to hold long slices: both first blocks of every wave are then read
      // before the slice length arrives (rows past a shorter slice are read
      // for nothing, never used).
      const bool spec2 = ring == 0 && (int64_t)L_cap >= (int64_t)DEC_SPEC2_ROWS * nw;
#define SCKV_DECODE_LAUNCH(DD, NWW, SP)                                                          \
  decode_mfma_kernel<DD, NWW, true, SP><<<slices, NWW * 64, 0, stream>>>(                         \
      qq, kn, vn, kc, vc, kv_len, cur_tok, vu, pos, L_meta, H, L_cap, qs, rotate, tab, part, 1,  \
      slices, L_cap, out, status, ring)
      constexpr int D1 = D <= 64 ? D : 64;  // nw == 1 only where D <= 64
      if (nw == 1 && spec2) SCKV_DECODE_LAUNCH(D1, 1, true);
      else if (nw == 1) SCKV_DECODE_LAUNCH(D1, 1, false);
      else if (nw == 2 && spec2) SCKV_DECODE_LAUNCH(D, 2, true);
      else if (nw == 2) SCKV_DECODE_LAUNCH(D, 2, false);
      else if (spec2) SCKV_DECODE_LAUNCH(D, 4, true);
      else SCKV_DECODE_LAUNCH(D, 4, false);
#undef SCKV_DECODE_LAUNCH
    } else {
      if (narrow)
        decode_chunk_kernel<T, D, 256, true><<<slices, 256, 0, stream>>>(
            qq, kn, vn, kc, vc, kv_len, cur_tok, vu, pos, L_meta, H, L_cap, qs, rotate, tab, part,
            1, slices, L_cap, out, status);
      else
        decode_chunk_kernel<T, D, 512, true><<<slices, 512, 0, stream>>>(
            qq, kn, vn, kc, vc, kv_len, cur_tok, vu, pos, L_meta, H, L_cap, qs, rotate, tab, part,
            1, slices, L_cap, out, status);
    }
    return hip_check(hipGetLastError(), "compacted_decode_attn: launch");
  }
  const int nc = n_chunks(L_cap);
  const int n_work = slices * nc;
  if constexpr (sizeof(T) == 2)
    decode_mfma_kernel<D, 4, false><<<n_work, 256, 0, stream>>>(
        qq, kn, vn, kc, vc, kv_len, cur_tok, vu, pos, L_meta, H, L_cap, qs, rotate, tab, part, nc,
        n_work, DEC_CH, out, status, ring);
  else
    decode_chunk_kernel<T, D, DEC_THREADS, false><<<n_work, DEC_THREADS, 0, stream>>>(
        qq, kn, vn, kc, vc, kv_len, cur_tok, vu, pos, L_meta, H, L_cap, qs, rotate, tab, part, nc,
        n_work, DEC_CH, out, status);
  int rc = hip_check(hipGetLastError(), "compacted_decode_attn: chunk launch");
  if (rc) return rc;
  decode_combine_kernel<T, D><<<slices, 64, 0, stream>>>(vn, kv_len, cur_tok, vu, L_meta, H, L_cap,
                                                          part, nc, DEC_CH, out, status, ring);
  return hip_check(hipGetLastError(), "compacted_decode_attn: combine launch");
}

}  // namespace sckv

using namespace sckv;

extern "C" size_t sckv_decode_workspace_bytes(int32_t b, int32_t H, int32_t L_cap, int32_t d_head) {
  if (b <= 0 || H <= 0 || L_cap <= 0 || d_head <= 0) return 0;
  return (size_t)b * H * n_chunks(L_cap) * (d_head + 2) * sizeof(float);
}

extern "C" int local_decode_attn(const void* q, const void* k_new, const void* v_new,
                                 void* k_cache, void* v_cache, int32_t W, const int32_t* cur_tok,
                                 const int32_t* vu, const int32_t* pos, int32_t L_meta, void* o,
                                 int32_t b, int32_t H, int32_t L_cap, int32_t d_head,
                                 sckv_dtype dt, float scale, float rope_theta, void* ws,
                                 size_t ws_bytes, int32_t* status, hipStream_t stream) {
  clear_error();
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !cur_tok || !vu || !o || !ws)
    return fail(SCKV_EINVAL, "local_decode_attn: null pointer");
  if (dt != SCKV_BF16) return fail(SCKV_EUNSUP, "local_decode_attn: bf16 only");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, "local_decode_attn: d_head must be 64 or 80");
  // W < L_cap: the W ring rows and the new token make W + 1 <= L_cap rows of
  // work, the most the launch and the workspace are sized for
  if (b <= 0 || H <= 0 || L_cap <= 0 || L_meta <= 0 || W <= 0 || W >= L_cap)
    return fail(SCKV_EINVAL, "local_decode_attn: need 0 < W < L_cap and positive sizes");
  if ((int64_t)b * H * n_chunks(L_cap) > 0x7fffffff)
    return fail(SCKV_EUNSUP, "local_decode_attn: b*H*chunks too large");
  if (!(scale > 0.f) || std::isinf(scale)) return fail(SCKV_EINVAL, "local_decode_attn: scale must be finite and > 0");
  if (!(rope_theta >= 0.f) || std::isinf(rope_theta))
    return fail(SCKV_EINVAL, "local_decode_attn: rope_theta must be finite and >= 0");
  if (rope_theta > 0.f && !pos) return fail(SCKV_EINVAL, "local_decode_attn: null pos");
  if (ws_bytes < sckv_decode_workspace_bytes(b, H, L_cap, d_head))
    return fail(SCKV_EINVAL, "local_decode_attn: workspace too small");
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
      !aligned16(v_cache) || !aligned16(o) || !aligned16(ws))
    return fail(SCKV_EINVAL, "local_decode_attn: buffers must be 16-byte aligned");
  const int32_t* p = pos ? pos : vu;
  return d_head == 64
             ? launch_decode<uint16_t, 64>(q, k_new, v_new, k_cache, v_cache, nullptr, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream, W)
             : launch_decode<uint16_t, 80>(q, k_new, v_new, k_cache, v_cache, nullptr, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream, W);
}

// Host checks of compacted_decode_attn and its allocation-free variant
// (everything but the workspace); no HIP call is made here.
static int decode_checks(const char* W, const void* q, const void* k_new, const void* v_new,
                         const void* k_cache, const void* v_cache, const int32_t* kv_len,
                         const int32_t* cur_tok, const int32_t* vu, const int32_t* pos,
                         int32_t L_meta, const void* o, int32_t b, int32_t H, int32_t L_cap,
                         int32_t d_head, sckv_dtype dt, float scale, float rope_theta) {
  const std::string w(W);
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !kv_len || !cur_tok || !vu || !o)
    return fail(SCKV_EINVAL, w + ": null pointer");
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, w + ": unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, w + ": d_head must be 64 or 80");
  if (b <= 0 || H <= 0 || L_cap <= 0 || L_meta <= 0)
    return fail(SCKV_EINVAL, w + ": sizes must be positive");
  if ((int64_t)b * H * n_chunks(L_cap) > 0x7fffffff)
    return fail(SCKV_EUNSUP, w + ": b*H*chunks too large");
  if (!(scale > 0.f) || std::isinf(scale)) return fail(SCKV_EINVAL, w + ": scale must be finite and > 0");
  if (!(rope_theta >= 0.f) || std::isinf(rope_theta))
    return fail(SCKV_EINVAL, w + ": rope_theta must be finite and >= 0");
  if (rope_theta > 0.f && !pos) return fail(SCKV_EINVAL, w + ": null pos");
  if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) ||
      !aligned16(v_cache) || !aligned16(o))
    return fail(SCKV_EINVAL, w + ": buffers must be 16-byte aligned");
  return SCKV_OK;
}

static int decode_dispatch(const void* q, const void* k_new, const void* v_new, void* k_cache,
                           void* v_cache, const int32_t* kv_len, const int32_t* cur_tok,
                           const int32_t* vu, const int32_t* pos, int32_t L_meta, void* o,
                           int32_t b, int32_t H, int32_t L_cap, int32_t d_head, sckv_dtype dt,
                           float scale, float rope_theta, void* ws, int32_t* status,
                           hipStream_t stream) {
  const int32_t* p = pos ? pos : vu;  // pos is read only when rotating
  if (dt == SCKV_BF16)
    return d_head == 64
               ? launch_decode<uint16_t, 64>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream)
               : launch_decode<uint16_t, 80>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream);
  return d_head == 64
             ? launch_decode<float, 64>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream)
             : launch_decode<float, 80>(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, p, L_meta, o, b, H, L_cap, scale, rope_theta, ws, status, stream);
}

extern "C" int compacted_decode_attn(const void* q, const void* k_new, const void* v_new,
                                     void* k_cache, void* v_cache, const int32_t* kv_len,
                                     const int32_t* cur_tok, const int32_t* vu,
                                     const int32_t* pos, int32_t L_meta, void* o, int32_t b,
                                     int32_t H, int32_t L_cap, int32_t d_head, sckv_dtype dt,
                                     float scale, float rope_theta, void* ws, size_t ws_bytes,
                                     int32_t* status, hipStream_t stream) {
  clear_error();
  const char* W = "compacted_decode_attn";
  int rc = decode_checks(W, q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos, L_meta,
                         o, b, H, L_cap, d_head, dt, scale, rope_theta);
  if (rc) return rc;
  if (!ws) return fail(SCKV_EINVAL, "compacted_decode_attn: null pointer");
  if (ws_bytes < sckv_decode_workspace_bytes(b, H, L_cap, d_head))
    return fail(SCKV_EINVAL, "compacted_decode_attn: workspace too small");
  if (!aligned16(ws)) return fail(SCKV_EINVAL, "compacted_decode_attn: buffers must be 16-byte aligned");
  return decode_dispatch(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos, L_meta, o, b,
                         H, L_cap, d_head, dt, scale, rope_theta, ws, status, stream);
}

// ---------------------------------------------------------------------------
// The same decode step without any allocation: the split-K partials go to a
// file-scope device array instead of a caller workspace.  Each device that
// runs the library holds its own copy of the array from module load until
// the process ends; its device address is looked up once per device (the
// array's name in host code is only a stand-in for that address) and kept.
// Every call on a device shares that device's array and leaves its partials
// in it; nothing in it has to start at zero (the merge reads only the chunk
// partials the same call wrote).  Calls that overlap on one device race.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char scratch[SCKV_NOALLOC_SCRATCH_BYTES];

constexpr int NOALLOC_MAX_DEVICES = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[NOALLOC_MAX_DEVICES];  // per device, set once

static int scratch_address(void** out) {
  int dev = -1;
  int rc = hip_check(hipGetDevice(&dev), "compacted_decode_attn_noalloc: hipGetDevice");
  if (rc) return rc;
  if (dev < 0 || dev >= NOALLOC_MAX_DEVICES)
    return fail(SCKV_EUNSUP, "compacted_decode_attn_noalloc: device index above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    rc = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)),
                   "compacted_decode_attn_noalloc: hipGetSymbolAddress(scratch)");
    if (rc) return rc;
    if (!p || !aligned16(p))
      return fail(SCKV_EHIP, "compacted_decode_attn_noalloc: scratch array has no usable address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SCKV_OK;
}

extern "C" int compacted_decode_attn_noalloc(const void* q, const void* k_new, const void* v_new,
                                             void* k_cache, void* v_cache, const int32_t* kv_len,
                                             const int32_t* cur_tok, const int32_t* vu,
                                             const int32_t* pos, int32_t L_meta, void* o,
                                             int32_t b, int32_t H, int32_t L_cap, int32_t d_head,
                                             sckv_dtype dt, float scale, float rope_theta,
                                             int32_t* status, hipStream_t stream) {
  clear_error();
  const char* W = "compacted_decode_attn_noalloc";
  int rc = decode_checks(W, q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos, L_meta,
                         o, b, H, L_cap, d_head, dt, scale, rope_theta);
  if (rc) return rc;
  // only the split launch (fewer than DEC_SINGLE_MIN slices) writes partials
  const size_t need = (int64_t)b * H >= DEC_SINGLE_MIN
                          ? 0 : sckv_decode_workspace_bytes(b, H, L_cap, d_head);
  if (need > SCKV_NOALLOC_SCRATCH_BYTES)
    return fail(SCKV_EUNSUP, std::string(W) + ": the split-K partials need " +
                                 std::to_string(need) + " bytes, more than the " +
                                 std::to_string((size_t)SCKV_NOALLOC_SCRATCH_BYTES) +
                                 "-byte scratch array (use compacted_decode_attn with a workspace)");
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc) return rc;
  return decode_dispatch(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos, L_meta, o, b,
                         H, L_cap, d_head, dt, scale, rope_theta, ws, status, stream);
}
