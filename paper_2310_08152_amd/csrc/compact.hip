// Freeing the key/value rows of closed spans: stable stream compaction of the
// (M, 2, b, H, L_cap, d) cache.  Section 3, "Manipulating Key-Value Memory for
// Inference-time Compression" (the memory of enclosed tokens is freed) with
// the cache layout of Section 2.
//
// Two kernels:
//   scan : one workgroup per sequence; keep flags from the span metadata, an
//          exclusive prefix sum (wave ballot + mbcnt, wave totals in LDS) that
//          gives every surviving row its new index; rewrites tok_idx/pos_ids
//          in place and emits kept_src_row.
//   move : one workgroup per (layer, k/v, sequence, head) slice; moves the
//          surviving rows to their new index, 16 bytes per lane, in chunks
//          that read everything before writing anything.  A row never moves
//          up (new index <= old index), so chunks taken in ascending order
//          never overwrite a row a later chunk still has to read.
#include "sckv_common.h"

namespace sckv {

constexpr int SCAN_THREADS = 256;
constexpr int MOVE_THREADS = 256;

__global__ __launch_bounds__(SCAN_THREADS) void compact_scan_kernel(
    int32_t* __restrict__ kv_len, int32_t* __restrict__ tok_idx, int32_t* __restrict__ pos_ids,
    const int32_t* __restrict__ next_tok, const int32_t* __restrict__ vu, int32_t L_meta,
    int32_t L_cap, int32_t* __restrict__ kept_src) {
  const int s = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  __shared__ int wave_cnt[SCAN_THREADS / 64];
  int n_old = kv_len[s];
  n_old = n_old < 0 ? 0 : (n_old > L_cap ? L_cap : n_old);
  const int P = next_tok[s];
  int32_t* tok = tok_idx + (int64_t)s * L_cap;
  int32_t* pp = pos_ids + (int64_t)s * L_cap;
  int32_t* ks = kept_src + (int64_t)s * L_cap;
  const int32_t* vus = vu + (int64_t)s * L_meta;
  int carry = 0;
  for (int base = 0; base < n_old; base += SCAN_THREADS) {
    const int row = base + tid;
    const bool valid = row < n_old;
    int t = 0, p = 0;
    bool keep = false;
    if (valid) {
      t = tok[row];
      p = pp[row];
      if (t < 0 || t >= L_meta) {
        keep = true;
      } else {
        const int v = vus[t];
        keep = (v != t) && (v >= P);
      }
    }
    wait_vmem();  // every read of this chunk has landed before any write below
    const uint64_t m = __ballot(keep);
    if ((tid & 63) == 0) wave_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = carry, total = 0;
#pragma unroll
    for (int w = 0; w < SCAN_THREADS / 64; ++w) {
      const int c = wave_cnt[w];
      if (w < wave) off += c;
      total += c;
    }
    if (keep) {
      const int rank = off + mask_rank(m);
      tok[rank] = t;
      pp[rank] = p;
      ks[rank] = row;
    }
    carry += total;
    __syncthreads();
  }
  for (int r = carry + tid; r < L_cap; r += SCAN_THREADS) ks[r] = -1;
  __syncthreads();  // every thread has read kv_len[s]
  if (tid == 0) kv_len[s] = carry;
}

// first rank r in [0, n) with ks[r] != r (n if none); ks[r] - r is
// non-decreasing, so the predicate is monotone.  Two rounds of probes.
__device__ int first_moving_rank(const int32_t* __restrict__ ks, int n, int* sh) {
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  if (n <= 0) return 0;
  const int S = (n + MOVE_THREADS - 1) / MOVE_THREADS;  // segment length
  // first pass: probe the last rank of every segment
  int seg_end = tid * S + S - 1;
  if (seg_end > n - 1) seg_end = n - 1;
  const bool moved = (tid * S < n) && (ks[seg_end] != seg_end);
  const uint64_t m1 = __ballot(moved);
  if ((tid & 63) == 0) sh[wave] = m1 ? (wave * 64 + __builtin_ctzll(m1)) : 0x7fffffff;
  __syncthreads();
  int t0 = 0x7fffffff;
  for (int w = 0; w < MOVE_THREADS / 64; ++w) t0 = min(t0, sh[w]);
  __syncthreads();
  if (t0 == 0x7fffffff) return n;
  // second pass: probe every rank of segment t0 (S <= MOVE_THREADS when n <= 65536)
  const int r = t0 * S + tid;
  const bool moved2 = (tid < S) && (r < n) && (ks[r] != r);
  const uint64_t m2 = __ballot(moved2);
  if ((tid & 63) == 0) sh[wave] = m2 ? (wave * 64 + __builtin_ctzll(m2)) : 0x7fffffff;
  __syncthreads();
  int t1 = 0x7fffffff;
  for (int w = 0; w < MOVE_THREADS / 64; ++w) t1 = min(t1, sh[w]);
  __syncthreads();
  return t1 == 0x7fffffff ? n : t0 * S + t1;
}

template <int ROWB, int U>
__global__ __launch_bounds__(MOVE_THREADS) void compact_move_kernel(
    char* kv, char* kv_out, int32_t b, int32_t H, int32_t L_cap,
    const int32_t* __restrict__ kv_len, const int32_t* __restrict__ kept_src) {
  constexpr int PPR = ROWB / 16;  // 16-byte pieces per row
  __shared__ int sh[MOVE_THREADS / 64];
  const int64_t slice = blockIdx.x;
  const int s = (int)((slice / H) % b);
  const int n = kv_len[s];
  const int32_t* ks = kept_src + (int64_t)s * L_cap;
  const char* src = kv + slice * (int64_t)L_cap * ROWB;
  char* dst = (kv_out ? kv_out : kv) + slice * (int64_t)L_cap * ROWB;
  const int f = kv_out ? 0 : first_moving_rank(ks, n, sh);
  const int64_t total = (int64_t)(n - f) * PPR;
  const int tid = threadIdx.x;
  for (int64_t c = 0; c < total; c += (int64_t)U * MOVE_THREADS) {
    u32x4 val[U];
    int drow[U], dseg[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t piece = c + (int64_t)u * MOVE_THREADS + tid;
      drow[u] = -1;
      if (piece < total) {
        const int r = f + (int)(piece / PPR);
        const int sg = (int)(piece % PPR);
        drow[u] = r;
        dseg[u] = sg;
        val[u] = ld16(src + (int64_t)ks[r] * ROWB + sg * 16);
      }
    }
    wait_vmem();
    __syncthreads();  // all reads of this chunk are done before any write
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (drow[u] >= 0) st16(dst + (int64_t)drow[u] * ROWB + dseg[u] * 16, val[u]);
  }
}

}  // namespace sckv

using namespace sckv;

extern "C" int kv_compact(void* kv, void* kv_out, int32_t M, int32_t b, int32_t H, int32_t L_cap,
                          int32_t d_head, sckv_dtype dt, int32_t* kv_len, int32_t* tok_idx,
                          int32_t* pos_ids, const int32_t* next_tok, const int32_t* vu,
                          int32_t L_meta, int32_t* kept_src_row, hipStream_t stream) {
  clear_error();
  if (!kv || !kv_len || !tok_idx || !pos_ids || !next_tok || !vu || !kept_src_row)
    return fail(SCKV_EINVAL, "kv_compact: null pointer");
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, "kv_compact: unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, "kv_compact: d_head must be 64 or 80");
  if (M <= 0 || b <= 0 || H <= 0 || L_cap <= 0 || L_meta <= 0)
    return fail(SCKV_EINVAL, "kv_compact: sizes must be positive");
  if (L_cap > 65536) return fail(SCKV_EUNSUP, "kv_compact: L_cap above 65536");
  if (kv_out == kv) return fail(SCKV_EINVAL, "kv_compact: kv_out must differ from kv (pass null for in place)");
  if (!aligned16(kv) || (kv_out && !aligned16(kv_out)))
    return fail(SCKV_EINVAL, "kv_compact: cache buffers must be 16-byte aligned");
  const int64_t slices = (int64_t)M * 2 * b * H;
  if (slices > 0x7fffffff) return fail(SCKV_EUNSUP, "kv_compact: too many slices");
  compact_scan_kernel<<<b, SCAN_THREADS, 0, stream>>>(kv_len, tok_idx, pos_ids, next_tok, vu,
                                                      L_meta, L_cap, kept_src_row);
  int rc = hip_check(hipGetLastError(), "kv_compact: scan launch");
  if (rc) return rc;
  const int rowb = d_head * elem_bytes(dt);
  char* a = static_cast<char*>(kv);
  char* o = static_cast<char*>(kv_out);
  const unsigned g = (unsigned)slices;
  switch (rowb) {
    case 128: compact_move_kernel<128, 8><<<g, MOVE_THREADS, 0, stream>>>(a, o, b, H, L_cap, kv_len, kept_src_row); break;
    case 160: compact_move_kernel<160, 8><<<g, MOVE_THREADS, 0, stream>>>(a, o, b, H, L_cap, kv_len, kept_src_row); break;
    case 256: compact_move_kernel<256, 8><<<g, MOVE_THREADS, 0, stream>>>(a, o, b, H, L_cap, kv_len, kept_src_row); break;
    case 320: compact_move_kernel<320, 8><<<g, MOVE_THREADS, 0, stream>>>(a, o, b, H, L_cap, kv_len, kept_src_row); break;
    default: return fail(SCKV_EUNSUP, "kv_compact: unsupported row size");
  }
  return hip_check(hipGetLastError(), "kv_compact: move launch");
}
