// Causal attention under the <CL>/<CR> span-exclusion mask (prefill).
// Section 1 (tokens after a <CR> do not attend to the tokens its span
// encloses) and Section 3.1 (<CL> attends only to itself; normal tokens attend
// to earlier <CR> and normal tokens).
//
// With vu[] as in sckv.h, row i may attend to column j iff
//   j <= i <= vu[j]  and  (vu[i] != i or j == i).
//
// plan kernel: for every (sequence, 128-row query block [I, I+128)) the list
//   of key columns j < I+128 with vu[j] >= I, i.e. the columns at least one
//   row of the block may see, in ascending order, packed as
//   j | min(vu[j]-I, 255) << 24.  Columns hidden from the whole block (closed
//   spans, <CL>s before the block) are not in the list and are never read.
//   It then summarises each 64-entry tile of the list (first and last token,
//   smallest rank, valid entries), so the main kernel stages a tile without
//   reductions of its own.
// main kernel: one workgroup per (sequence, head, query block), 4 waves of 32
//   query rows.  Key/value rows named by the list are gathered 64 at a time
//   into LDS (double buffered for bf16); S^T = K Q^T and O^T += V^T P^T run
//   on 32x32 MFMA tiles (bf16 inputs, fp32 accumulation; fp32 inputs use the
//   fp32 MFMA), with an online softmax per query held in the lane that owns
//   the query's column.  Element masks are applied only on tiles that are
//   not entirely visible to a wave; a tile entirely in a wave's future is
//   skipped.  A <CL> row's output is its own value row (it sees only itself),
//   written directly in the epilogue.
//
// Cached variant (block-wise prompt processing, Section 3 "Manipulating
// Key-Value Memory": enclosed tokens are freed block by block when a prompt
// does not fit): the queries are a block of the prompt, tokens tok0 .. tok0+nq-1,
// and the keys are the rows of a cache, row r holding token tok[r] (rows of
// earlier blocks that survived compaction, then the block's own rows from
// row0).  The plan lists cache rows instead of columns, with the same
// visibility rule applied to their tokens; the kernel gathers by row and
// masks by token.
#include <math.h>

#include <cmath>
#include <type_traits>

#include "sckv_common.h"

namespace sckv {

// waves per workgroup, 32 query rows each (six and eight waves, sharing each
// staged tile among more rows, measured 20-45% slower than four)
constexpr int PF_WAVES = 4;
constexpr int PF_BQ = 32 * PF_WAVES;
constexpr int PF_BK = 64;
// a block's list has room for at least two tiles (its first two are loaded early)
static_assert(PF_BQ >= 2 * PF_BK, "list of at least two tiles");
constexpr int PF_THREADS = 64 * PF_WAVES;
// (sequence, head) slices whose query blocks are ordered together,
// heaviest first (a dispatch simulation over the two prompt shapes puts
// groups of 8 within 3-6% of an ideal balance, against 9-18% for one slice)
constexpr int PF_GROUP = 8;
constexpr uint32_t PF_NONE = 0x00ffffffu;  // list entry of a padding column
constexpr float PF_LOG2E = 1.4426950408889634f;
// The running maximum of a query row is only moved (and the accumulators
// rescaled) when a tile's maximum exceeds it by more than this many powers of
// two; until then probabilities are taken relative to the older, smaller
// maximum, which is exact and keeps them below 2^PF_RESCALE.
constexpr float PF_RESCALE = 8.f;

// Cached variant's arguments (unused by the plain prefill).
struct PfCached {
  const int32_t* row0;   // [b] cache row of the block's first query token
  const int32_t* tok;    // [b][L_cap] token held by each cache row
  uint32_t* rows;        // plan output: cache row of each list entry
  int32_t tok0;          // token of the block's first query
  int32_t L_cap;
  int32_t* status;       // nullable: SCKV_STATUS_CAP for a block that does not fit
};

// Summary of one 64-entry tile of a list, written by the plan kernel: first
// and last listed token, smallest rank byte | valid entries << 8, and the row
// a padding slot of the tile repeats (the last valid entry's row).
struct TileSum {
  int32_t jmin, jmax, vr_n, pad_row;
};

// Plain: columns j < min(I+128, L) with token j.  Cached: cache rows
// r < row0 + min(I_loc+128, nq) with token tok[r], where I_loc is the query
// block's first local row and I = tok0 + I_loc its first token.
template <bool CACHED>
__global__ __launch_bounds__(256) void prefill_plan_kernel(const int32_t* __restrict__ vu,
                                                           int32_t L_meta, int32_t L, int32_t n_qt,
                                                           int32_t L_pad,
                                                           uint32_t* __restrict__ list,
                                                           int32_t* __restrict__ count,
                                                           TileSum* __restrict__ info,
                                                           PfCached cc) {
  const int qt = blockIdx.x;
  const int s = blockIdx.y;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int I_loc = qt * PF_BQ;
  int I = I_loc, jend = min(I_loc + PF_BQ, L);
  if constexpr (CACHED) {
    I = cc.tok0 + I_loc;
    const int r0 = cc.row0[s];
    const bool fits = r0 >= 0 && (int64_t)r0 + L <= cc.L_cap;
    jend = fits ? r0 + min(I_loc + PF_BQ, L) : 0;
  }
  const int32_t* v = vu + (int64_t)s * L_meta;
  uint32_t* out = list + ((int64_t)s * n_qt + qt) * L_pad;
  __shared__ int wave_cnt[4];
  int carry = 0;
  for (int base = 0; base < jend; base += 256) {
    const int j = base + tid;
    bool ok = false;
    uint32_t e = 0;
    if (j < jend) {
      // the column's token: the row itself, or the token a cache row holds
      // (a row whose token lies outside [0, L_meta) is never listed)
      const int t = CACHED ? cc.tok[(int64_t)s * cc.L_cap + j] : j;
      if (!CACHED || (t >= 0 && t < L_meta)) {
        const int x = v[t];
        ok = x >= I;
        const int64_t rel = (int64_t)x - I;
        e = (uint32_t)t | ((uint32_t)(rel > 255 ? 255 : rel) << 24);
      }
    }
    const uint64_t m = __ballot(ok);
    if ((tid & 63) == 0) wave_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = carry, total = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = wave_cnt[w];
      if (w < wave) off += c;
      total += c;
    }
    if (ok) {
      out[off + mask_rank(m)] = e;
      if constexpr (CACHED) cc.rows[((int64_t)s * n_qt + qt) * L_pad + off + mask_rank(m)] = j;
    }
    carry += total;
    __syncthreads();
  }
  if (tid == 0) count[(int64_t)s * n_qt + qt] = carry;

  // tile summaries: wave w takes tiles w, w+4, ... of the list just written
  // (the barrier that ended the last round orders those writes before these
  // reads)
  const int lane = tid & 63;
  const uint32_t* rws = CACHED ? cc.rows + ((int64_t)s * n_qt + qt) * L_pad : nullptr;
  TileSum* sum = info + ((int64_t)s * n_qt + qt) * (L_pad / 64);
  for (int t = wave; t * 64 < carry; t += 4) {
    const int nvalid = min(64, carry - t * 64);
    const bool in = lane < nvalid;
    const uint32_t e = in ? out[t * 64 + lane] : PF_NONE;
    int vr = in ? (int)(e >> 24) : 255;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) vr = min(vr, __shfl_xor(vr, off, 64));
    const int jmin = __shfl((int)(e & 0x00ffffffu), 0, 64);
    const int jmax = __shfl((int)(e & 0x00ffffffu), nvalid - 1, 64);
    int pad = jmax;
    if constexpr (CACHED) pad = __shfl(in ? (int)rws[t * 64 + lane] : 0, nvalid - 1, 64);
    if (lane == 0) sum[t] = TileSum{jmin, jmax, vr | (nvalid << 8), pad};
  }
}

// ---------------------------------------------------------------------------
// tile geometry per element type
// ---------------------------------------------------------------------------
template <typename T, int D> struct PfCfg;

template <int D> struct PfCfg<uint16_t, D> {
  static constexpr int NBUF = 2;
  static constexpr int DP = (D + 31) / 32 * 32;     // value columns padded to whole 32-row MFMA blocks
  static constexpr int KP = D + 8;                  // K tile: [64][KP] bf16 (one 16-byte pad slot)
  // V tile: [64][VP] bf16, row-major like K; the PV operand is read with the
  // transposing LDS read.  With a ones row (D = 80) the pitch is 192 bytes,
  // which puts the four rows one transposing read touches in disjoint groups
  // of 16 banks.  At D = 64 the rows are unpadded (128 bytes) and the
  // 16-byte pieces of a row are swizzled instead: logical piece p of row r
  // sits in slot p ^ (4 * bit 1 of r), which spreads the rows of one
  // transposing read over the banks the same way in two thirds of the space.
  static constexpr bool VSWZ = (D == 64);
  static constexpr int VP = VSWZ ? D : 96;
  static constexpr int NB = D == 64 ? 1 : 2;        // 32-key blocks per softmax step
  static_assert(DP <= VP, "value tile pitch");
  static constexpr int E = 8;                       // elements per 16-byte slot
  static constexpr int KSTEPS = D / 16;
};

template <int D> struct PfCfg<float, D> {
  static constexpr int NBUF = 1;
  static constexpr bool VSWZ = false;
  static constexpr int NB = 2;
  static constexpr int DP = (D + 31) / 32 * 32;
  static constexpr int KP = D + 4;                  // K tile: [64][KP] f32
  static constexpr int VP = DP + 8;                 // V tile: [64][VP] f32 (row-major)
  static constexpr int E = 4;
  static constexpr int KSTEPS = D / 2;
};

// Row slots of a staged tile.  Rows are copied global -> LDS by the
// direct-to-LDS load (16 bytes per lane, lane i of an instruction writes
// slot base+i), so a tile is a whole number of 1 KiB blocks of 64 slots.
template <typename T, int D>
struct PfTile {
  using C = PfCfg<T, D>;
  static constexpr int PPR = D / C::E;                         // data slots per row
  static constexpr int KSLOT = C::KP * (int)sizeof(T) / 16;    // slots per K row
  static constexpr int VSLOT = C::VP * (int)sizeof(T) / 16;    // slots per V row
  static_assert(C::KP * sizeof(T) % 16 == 0 && C::VP * sizeof(T) % 16 == 0, "slot pitch");
  static constexpr int KBYTES = PF_BK * KSLOT * 16;            // == KSLOT KiB
  static constexpr int VBYTES = PF_BK * VSLOT * 16;
};

struct TileInfo {
  int jmin, jmax, vrmin, nvalid;
};

// maximum of x over lanes l and l^32: one lane swap between the two
// 32-lane halves of the wave (v_permlane32_swap leaves each lane holding
// the pair's two values, one in each result)
__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return a > b ? a : b;
}

constexpr int PF_ER = 4;  // ring of list entries: tile kt+2 is fetched while kt is computed

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// ---------------------------------------------------------------------------
// main kernel
// ---------------------------------------------------------------------------
template <typename T, int D, bool CACHED>
__device__ __forceinline__ void prefill_attn_body(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, T* __restrict__ o,
    int32_t H, int32_t L, int64_t qs, int64_t kvs, int64_t os, float c2,
    const int32_t* __restrict__ vu, int32_t L_meta, const uint32_t* __restrict__ list,
    const int32_t* __restrict__ count, const TileSum* __restrict__ info, int32_t n_qt,
    int32_t L_pad, int32_t n_work, PfCached cc) {
  using C = PfCfg<T, D>;
  using TL = PfTile<T, D>;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int NDB = C::DP / 32;                           // output d blocks

  // Separate objects per buffer: the compiler then knows that a
  // direct-to-LDS load into one buffer does not feed reads of the other.
  __shared__ __align__(1024) char kbuf0[TL::KBYTES];
  __shared__ __align__(1024) char vbuf0[TL::VBYTES];
  __shared__ __align__(1024) char kbuf1[C::NBUF == 2 ? TL::KBYTES : 1024];
  __shared__ __align__(1024) char vbuf1[C::NBUF == 2 ? TL::VBYTES : 1024];
  __shared__ uint32_t ent_ring[PF_ER][PF_BK];
  __shared__ int32_t row_ring[PF_ER][PF_BK];  // bare row index per entry
  __shared__ TileInfo info_ring[PF_ER];

  // Work order.  Workgroup x is dispatched to XCD x mod 8, and each XCD takes
  // a contiguous range of work items in dispatch order, so the items of a
  // group of PF_GROUP consecutive (sequence, head) slices share that XCD's
  // L2.  Inside a group the items go heaviest first: every head's last
  // query block (the most visible keys), then every head's block before it,
  // and so on, so that the light blocks fill the end of the launch instead
  // of one slice's heavy block running alone there.
  const int x = blockIdx.x;
  const int xcd = x & 7, idx = x >> 3;
  const int qn = n_work >> 3, rem = n_work & 7;
  const int work = xcd * qn + min(xcd, rem) + idx;
  const int nbh = n_work / n_qt;
  const int grp = work / (PF_GROUP * n_qt);
  const int gsz = min(PF_GROUP, nbh - grp * PF_GROUP);
  const int in_grp = work - grp * PF_GROUP * n_qt;
  const int bh = grp * PF_GROUP + in_grp % gsz;
  const int qt = n_qt - 1 - in_grp / gsz;
  const int s = bh / H;
  // query rows are local (0 .. L-1); their tokens start at tok0 (cached) or 0
  const int tok0 = CACHED ? cc.tok0 : 0;
  const int I_loc = qt * PF_BQ;
  const int I = tok0 + I_loc;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int g = lane >> 5;
  const int Iw_loc = I_loc + wave * 32;
  const int Iw = I + wave * 32;
  const int qrow = Iw_loc + l32;  // local query row
  const int qtok = Iw + l32;      // its token
  const bool wave_live = Iw_loc < L;

  const T* qb = q + (int64_t)bh * qs;
  const T* kb = k + (int64_t)bh * kvs;
  const T* vb = v + (int64_t)bh * kvs;
  const uint32_t* ents = list + ((int64_t)s * n_qt + qt) * L_pad;
  const uint32_t* rws = CACHED ? cc.rows + ((int64_t)s * n_qt + qt) * L_pad : nullptr;
  const TileSum* tsum = info + ((int64_t)s * n_qt + qt) * (L_pad / 64);
  int own_row0 = 0;  // cache row of local query row 0
  if constexpr (CACHED) {
    own_row0 = cc.row0[s];
    if (own_row0 < 0 || (int64_t)own_row0 + L > cc.L_cap) {
      // the block's rows are not in the cache: NaN outputs, nothing read
      if (cc.status && tid == 0 && qt == 0 && (bh % H) == 0) atomicOr(cc.status, SCKV_STATUS_CAP);
      if (wave_live && qrow < L) {
        T* orow = o + (int64_t)bh * os + (int64_t)qrow * D;
        for (int e = g; e < D; e += 2) {
          if constexpr (sizeof(T) == 2) orow[e] = (T)0x7fc0;
          else orow[e] = NAN;
        }
      }
      return;
    }
  }
  // clamped into the list, so that a workspace holding no valid plan (a
  // caller's mistake with the planned entry point) reads nothing outside it
  const int n_vis = min(max(count[(int64_t)s * n_qt + qt], 0), L_pad);
  const int nt = (n_vis + PF_BK - 1) / PF_BK;

  // Padding value rows/columns are written once and never again.  For bf16
  // with padding, V^T row D is all ones, so the PV MFMA also produces each
  // query's probability sum (O^T row D) and no separate row sum is needed.
  constexpr bool ONES_SUM = BF && (C::DP != D);
  // Without padding (bf16, D = 64) the sums come from a 16x16x32 MFMA of the
  // probabilities against a 0/1 matrix: lane L's A operand is all ones when
  // bit 2 of L equals bit 4 of L, so D[4*(L/16) + j][L%16] adds the two
  // lanes that hold query L%32's probabilities (lanes q and q + 32 of the
  // 32x32x16 B operand), and every lane receives its own query's sum.
  constexpr bool MFMA_SUM = BF && !ONES_SUM;
  if constexpr (C::DP != D) {
    for (int b = 0; b < C::NBUF; ++b) {
      char* vbuf = b == 0 ? vbuf0 : vbuf1;
      if constexpr (BF) {
        uint16_t* vs = reinterpret_cast<uint16_t*>(vbuf);
        for (int i = tid; i < PF_BK * (C::DP - D); i += PF_THREADS) {
          const int c = D + i % (C::DP - D);
          vs[(i / (C::DP - D)) * C::VP + c] = (c == D) ? (uint16_t)0x3f80 : (uint16_t)0;
        }
      } else {
        float* vs = reinterpret_cast<float*>(vbuf);
        for (int i = tid; i < PF_BK * (C::DP - D); i += PF_THREADS)
          vs[(i / (C::DP - D)) * C::VP + D + i % (C::DP - D)] = 0.f;
      }
    }
  }

  // Q^T operand, held for the whole kernel
  using QReg = typename std::conditional<BF, bf16x8, float>::type;
  QReg qreg[C::KSTEPS];
#pragma unroll
  for (int kk = 0; kk < C::KSTEPS; ++kk) {
    if constexpr (BF) {
      u32x4 w = qrow < L ? ld16(qb + (int64_t)qrow * D + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      qreg[kk] = __builtin_bit_cast(bf16x8, w);
    } else {
      qreg[kk] = qrow < L ? qb[(int64_t)qrow * D + 2 * kk + g] : 0.f;
    }
  }

  // A <CL> row's output is its own value row.  It is copied here, where its
  // loads overlap the staging of the first tiles, rather than after the loop
  // (the epilogue then writes only the other rows).
  const bool is_cl = qrow < L && vu[(int64_t)s * L_meta + qtok] == qtok;
  T* const orow = o + (int64_t)bh * os + (int64_t)qrow * D;
  if (is_cl) {
    const T* vrow = vb + (int64_t)(own_row0 + qrow) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d0 = db * 32 + 8 * jj + 4 * g;
        if (d0 >= D) continue;
        if constexpr (BF) *reinterpret_cast<u32x2*>(orow + d0) = *reinterpret_cast<const u32x2*>(vrow + d0);
        else st16(orow + d0, ld16(vrow + d0));
      }
  }

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 lacc = {0.f, 0.f, 0.f, 0.f};

  // ---- staging: list entries run two tiles ahead through an LDS ring; the
  // key/value rows of tile kt+1 go global -> LDS by direct loads addressed
  // from the ring while tile kt is multiplied ----
  // a tile's list entries (wave 0's lanes), their cache rows (cached) and the
  // plan's summary of the tile, between their load and their ring slot
  struct Staged {
    uint32_t e;
    int r;
    TileSum s;
  };
  Staged stg = {PF_NONE, 0, {0, 0, 0, 0}};
  auto nvalid_of = [&](int kt) { return min(PF_BK, n_vis - kt * PF_BK); };
  // The loads do not depend on the list's length (tile kt < max(nt, 2) lies
  // inside the block's list of L_pad >= 128 entries), so the first tiles'
  // loads need not wait for the count; the length masks them when stored.
  auto load_entries = [&](int kt, Staged& st) {
    if (tid < PF_BK) {
      st.e = ents[kt * PF_BK + tid];
      if constexpr (CACHED) st.r = (int)rws[kt * PF_BK + tid];
    }
    if (wave == 0) st.s = tsum[kt];
  };
  // wave 0 writes the ring slot of tile kt from the entries and the plan's
  // summary of the tile
  auto store_entries = [&](int kt, const Staged& st) {
    const bool in = lane < nvalid_of(kt);
    const uint32_t ereg = in ? st.e : PF_NONE;
    const int rreg = in ? st.r : 0;
    const TileSum sreg = st.s;
    const int slot = kt % PF_ER;
    if (wave == 0) {
      const int vr_n = __builtin_amdgcn_readfirstlane(sreg.vr_n);
      const int nvalid = vr_n >> 8;
      ent_ring[slot][lane] = ereg;
      // a padding row of the tile repeats the last valid row (its score is
      // masked, so any finite row will do)
      const int row = CACHED ? rreg : (int)(ereg & 0x00ffffffu);
      row_ring[slot][lane] = lane < nvalid ? row : __builtin_amdgcn_readfirstlane(sreg.pad_row);
      if (lane == 0) {
        TileInfo ti;
        ti.jmin = sreg.jmin;
        ti.jmax = sreg.jmax;
        ti.vrmin = vr_n & 255;
        ti.nvalid = nvalid;
        info_ring[slot] = ti;
      }
    }
  };
  // K and V of tile kt into kdst/vdst: slot sl = r*NSLOT + sg of a matrix
  // holds elements [sg*E, sg*E+E) of row r; pad slots are not written (they
  // keep their initial contents).  All row indices are read from the ring
  // first, then the copies are issued.  The indices come from row_ring, which
  // holds them bare: no masking of the packed entry happens on this path.
  constexpr int KRND = (TL::KSLOT + PF_WAVES - 1) / PF_WAVES;
  constexpr int VRND = (TL::VSLOT + PF_WAVES - 1) / PF_WAVES;
  // Copies go through buffer loads with an LDS destination: a 32-bit byte
  // offset per lane against a descriptor of the slice (reads past the slice
  // return zeros instead of faulting), the LDS block address in scalar
  // registers.  Each lane's tile row and piece offset per round are fixed
  // for the kernel and computed once here.
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const int slice_bytes = (int)min((int64_t)kvs * (int64_t)sizeof(T), (int64_t)0x7fffffff);
  const __amdgpu_buffer_rsrc_t krs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(kb), 0, slice_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(vb), 0, slice_bytes, 0x00020000);
  constexpr int ROWB = D * (int)sizeof(T);
  int k_row[KRND], k_off[KRND], v_row[VRND], v_off[VRND];
#pragma unroll
  for (int rnd = 0; rnd < KRND; ++rnd) {
    const int sl = (rnd * PF_WAVES + wave) * 64 + lane;
    const int sg = sl % TL::KSLOT;
    k_row[rnd] = min(sl / TL::KSLOT, PF_BK - 1);
    // a key row's pad slot is never read, so it is copied too (whatever the
    // 16 bytes after the row hold): no lane of a copy is masked off
    k_off[rnd] = sg * 16;
  }
#pragma unroll
  for (int rnd = 0; rnd < VRND; ++rnd) {
    const int sl = (rnd * PF_WAVES + wave) * 64 + lane;
    const int sg = sl % TL::VSLOT;
    v_row[rnd] = min(sl / TL::VSLOT, PF_BK - 1);
    int vpiece = sg;  // the logical piece slot sg holds
    if constexpr (BF) {
      if constexpr (C::VSWZ) vpiece = sg ^ (((v_row[rnd] >> 1) & 1) << 2);
    }
    // the value tile's pad slots hold the ones row and zeros (D = 80) and
    // must not be overwritten; without them (D = 64) every slot is data
    v_off[rnd] = sg < TL::PPR ? vpiece * 16 : -1;
  }
  auto dma_rows = [&](int kt, char* kdst, char* vdst) {
    const int32_t* rows = row_ring[kt % PF_ER];
    int kj[KRND], vj[VRND];
#pragma unroll
    for (int rnd = 0; rnd < KRND; ++rnd) kj[rnd] = rows[k_row[rnd]];
#pragma unroll
    for (int rnd = 0; rnd < VRND; ++rnd) vj[rnd] = rows[v_row[rnd]];
#pragma unroll
    for (int rnd = 0; rnd < KRND; ++rnd) {
      const int blk = rnd * PF_WAVES + wave_s;
      if (blk < TL::KSLOT)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lds_ptr_t)(kdst + blk * 1024), 16,
                                                 kj[rnd] * ROWB + k_off[rnd], 0, 0, 0);
    }
#pragma unroll
    for (int rnd = 0; rnd < VRND; ++rnd) {
      const int blk = rnd * PF_WAVES + wave_s;
      if (blk < TL::VSLOT && (TL::VSLOT == TL::PPR || v_off[rnd] >= 0))
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vrs, (lds_ptr_t)(vdst + blk * 1024), 16,
                                                 vj[rnd] * ROWB + v_off[rnd], 0, 0, 0);
    }
  };

  // Transposing-read addresses of the V^T operand, per 32-column block db
  // of the value tile: within each group of 16 lanes, lane j points at
  // V[kbase + j/4][dbase + 4*(j%4)]; the read hands lane i the four keys
  // kbase..kbase+3 of column dbase + i.  Offsets in elements from the tile
  // start; a step t of 16 keys adds (16 t) rows, its upper 8 keys 8 rows.
  int v_lane_off[NDB];
  {
    const int G = lane >> 4, j16 = lane & 15;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int col = 32 * db + 16 * (G & 1) + 4 * (j16 & 3);
      const int row = 4 * g + (j16 >> 2);  // bit 1 of the row is bit 1 of j16 >> 2
      if constexpr (BF && C::VSWZ)
        v_lane_off[db] = row * C::VP + (((col >> 3) ^ (((row >> 1) & 1) << 2)) << 3) + (col & 7);
      else
        v_lane_off[db] = row * C::VP + col;
    }
  }

  // summary of the tile being computed, read from the ring one step early
  // so that the step starts with its key reads
  TileInfo tcur;
  // A 64-key tile is weighed in softmax steps of NB 32-key blocks: scores
  // of the step, its online softmax, its share of the value product.  At
  // D = 64 a step is one block (32 keys), so only half a tile's scores and
  // probabilities are live at a time and four waves fit per SIMD; at D = 80
  // a step is the whole tile (measured faster there, at three waves either
  // way).
  constexpr int NB = C::NB;
  auto compute = [&](int kt, const char* kcur, const char* vcur) {
    const TileInfo ti = tcur;
    const uint32_t* tent = ent_ring[kt % PF_ER];
    if (wave_live && ti.jmin <= Iw + 31) {
      const bool full = ti.nvalid == PF_BK && ti.jmax <= Iw && ti.vrmin >= Iw + 31 - I;
      // With one 32-key block per step, the second block is skipped where
      // no row of this wave can see any of it: it lies past the list's end,
      // or (the list being in token order) its first token is later than the
      // wave's last row.
      bool skip2 = false;
      if constexpr (NB == 1) {
        const int j32 = __builtin_amdgcn_readfirstlane((int)(tent[32] & 0x00ffffffu));
        skip2 = ti.nvalid <= 32 || j32 > Iw + 31;
      }
#pragma unroll
      for (int st = 0; st < 2 / NB; ++st) {
        if (st == 1 && skip2) break;
        // ---- S^T = K Q^T for the step's key blocks, key step outer so that
        // consecutive matrix instructions write different accumulators ----
        f32x16 sacc[NB];
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i) sacc[kb][i] = 0.f;
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk) {
#pragma unroll
          for (int kb = 0; kb < NB; ++kb) {
            const int kb2 = st * NB + kb;
            if constexpr (BF) {
              const char* krow = kcur + ((kb2 * 32 + l32) * C::KP + g * 8 + kk * 16) * 2;
              const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(krow));
              sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], sacc[kb], 0, 0, 0);
            } else {
              const float* krow = reinterpret_cast<const float*>(kcur) + (kb2 * 32 + l32) * C::KP + g;
              sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(krow[2 * kk], qreg[kk], sacc[kb], 0, 0, 0);
            }
          }
        }
        // ---- element mask on tiles not entirely visible to this wave ----
        if (!full) {
          const int ir = qtok - I;
#pragma unroll
          for (int kb = 0; kb < NB; ++kb)
#pragma unroll
            for (int vv = 0; vv < 16; ++vv) {
              const int key = (st * NB + kb) * 32 + 8 * (vv >> 2) + 4 * g + (vv & 3);
              const uint32_t e = tent[key];
              const int j = (int)(e & 0x00ffffffu);
              const int vr = (int)(e >> 24);
              const bool vis = (j <= qtok) & (ir <= vr);
              sacc[kb][vv] = vis ? sacc[kb][vv] : -INFINITY;
            }
        }
        // ---- online softmax (log2 units), lazy rescaling ----
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
          for (int vv = 0; vv < 16; ++vv) mx = fmaxf(mx, sacc[kb][vv]);
        mx = max_across_halves(mx) * c2;
        const bool grow = mx > m_run + PF_RESCALE;
        if (__ballot(grow) != 0) {
          const float alpha = grow ? fast_exp2(m_run - mx) : 1.f;  // m_run == -inf gives 0
          if (grow) m_run = mx;
          if constexpr (MFMA_SUM) lacc *= alpha;
          else l_run *= alpha;
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
        }
        const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
          for (int vv = 0; vv < 16; ++vv) {
            const float p = fast_exp2(fmaf(sacc[kb][vv], c2, -m_use));
            sacc[kb][vv] = p;
            if constexpr (!ONES_SUM && !MFMA_SUM) rs += p;
          }
        if constexpr (!ONES_SUM && !MFMA_SUM) l_run += rs;
        // ---- O^T += V^T P^T over the step's keys, 16 at a time ----
        if constexpr (BF) {
          bf16x8 pb[2 * NB];
#pragma unroll
          for (int tt = 0; tt < 2 * NB; ++tt) {
            u32x4 w;
#pragma unroll
            for (int i = 0; i < 4; ++i)
              w[i] = pack_bf16x2(sacc[tt >> 1][8 * (tt & 1) + 2 * i], sacc[tt >> 1][8 * (tt & 1) + 2 * i + 1]);
            pb[tt] = __builtin_bit_cast(bf16x8, w);
          }
          if constexpr (MFMA_SUM) {
            const int ln = threadIdx.x & 63;
            const uint32_t one = (((ln >> 2) ^ (ln >> 4)) & 1) ? 0u : 0x3f803f80u;
            const bf16x8 ones_a = __builtin_bit_cast(bf16x8, u32x4{one, one, one, one});
#pragma unroll
            for (int tt = 0; tt < 2 * NB; ++tt)
              lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_a, pb[tt], lacc, 0, 0, 0);
          }
          const uint16_t* vs = reinterpret_cast<const uint16_t*>(vcur);
#pragma unroll
          for (int tt = 0; tt < 2 * NB; ++tt) {
            const int t = 2 * NB * st + tt;
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
              const s16x4 lo = lds_read_tr16(vs + v_lane_off[db] + (16 * t) * C::VP);
              const s16x4 hi = lds_read_tr16(vs + v_lane_off[db] + (16 * t + 8) * C::VP);
              const s16x8 vw = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
              oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw),
                                                                 pb[tt], oacc[db], 0, 0, 0);
            }
          }
        } else {
          const float* vs = reinterpret_cast<const float*>(vcur);
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int kb = 0; kb < NB; ++kb)
#pragma unroll
              for (int vv = 0; vv < 16; ++vv) {
                const int key = (st * NB + kb) * 32 + 8 * (vv >> 2) + 4 * g + (vv & 3);
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(vs[key * C::VP + db * 32 + l32],
                                                                sacc[kb][vv], oacc[db], 0, 0, 0);
              }
        }
      }
    }
  };

  // one tile: rows of kt+1 start moving, kt is multiplied, everything is
  // waited for, the ring advances
  auto iteration = [&](int kt, const char* kc, const char* vc, char* kn, char* vn) {
    if constexpr (C::NBUF == 2) {
      if (kt + 1 < nt) dma_rows(kt + 1, kn, vn);
    }
    if (kt + 2 < nt) load_entries(kt + 2, stg);
    compute(kt, kc, vc);
    if (kt + 1 < nt) tcur = info_ring[(kt + 1) % PF_ER];
    if constexpr (C::NBUF == 1) {
      __syncthreads();
      if (kt + 1 < nt) dma_rows(kt + 1, kn, vn);
    }
    wait_vmem();
    if (kt + 2 < nt) store_entries(kt + 2, stg);
    __syncthreads();
  };

  // tiles 0 and 1 staged with one round trip: both loads (issued without
  // waiting for the list's length) before either store
  {
    Staged st1 = {PF_NONE, 0, {0, 0, 0, 0}};
    load_entries(0, stg);
    load_entries(1, st1);
    store_entries(0, stg);
    if (nt > 1) store_entries(1, st1);
  }
  __syncthreads();
  dma_rows(0, kbuf0, vbuf0);
  wait_vmem();
  __syncthreads();
  tcur = info_ring[0];

  for (int kt = 0; kt < nt; kt += 2) {
    if constexpr (C::NBUF == 2) {
      iteration(kt, kbuf0, vbuf0, kbuf1, vbuf1);
      if (kt + 1 < nt) iteration(kt + 1, kbuf1, vbuf1, kbuf0, vbuf0);
    } else {
      iteration(kt, kbuf0, vbuf0, kbuf0, vbuf0);
      if (kt + 1 < nt) iteration(kt + 1, kbuf0, vbuf0, kbuf0, vbuf0);
    }
  }

  // ---- epilogue: normalise and write (<CL> rows were written at the start) ----
  if (!wave_live) return;
  float l_tot;
  if constexpr (ONES_SUM) {
    // O^T row D sits in d-block D/32, accumulator 8*((D%32)/8) of lane group 0
    static_assert((D % 32) % 8 == 0, "ones row must start a group of 8 rows");
    l_tot = __shfl(oacc[D / 32][4 * ((D % 32) / 8)], l32, 64);
  } else if constexpr (MFMA_SUM) {
    l_tot = lacc[0];
  } else {
    l_tot = l_run + __shfl_xor(l_run, 32, 64);
  }
  if (qrow >= L || is_cl) return;
  const float inv = 1.f / l_tot;
  // The output row's address is recomputed here from an opaque copy of the
  // lane index rather than kept from the start of the kernel: holding it
  // (and the lane's column offset) across the tile loop costs registers the
  // loop needs.
  int lane_e = threadIdx.x & 63;
  asm volatile("" : "+v"(lane_e));
  T* const orow_e = o + (int64_t)bh * os + (int64_t)(Iw_loc + (lane_e & 31)) * D + 4 * (lane_e >> 5);
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d0 = db * 32 + 8 * jj;
      if (d0 >= D) continue;  // D and d0 are multiples of 8
      if constexpr (BF) {
        u32x2 w;
        w[0] = pack_bf16x2(oacc[db][4 * jj] * inv, oacc[db][4 * jj + 1] * inv);
        w[1] = pack_bf16x2(oacc[db][4 * jj + 2] * inv, oacc[db][4 * jj + 3] * inv);
        *reinterpret_cast<u32x2*>(orow_e + d0) = w;
      } else {
        u32x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(oacc[db][4 * jj + i] * inv);
        st16(orow_e + d0, w);
      }
    }
}

// bf16 runs at four waves per SIMD at D = 64 (at most 128 registers; 36.9 KB
// of LDS per workgroup, so four workgroups share a CU) and at three at D = 80
// (at most 168 registers; 49 KB of LDS), each measured faster than one wave
// fewer; the fp32 variant (small parity cases) is not capped.
template <int D, bool CACHED>
__global__ __launch_bounds__(PF_THREADS) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 3))) void prefill_attn_kernel_bf16(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    uint16_t* __restrict__ o, int32_t H, int32_t L, int64_t qs, int64_t kvs, int64_t os, float c2,
    const int32_t* __restrict__ vu, int32_t L_meta, const uint32_t* __restrict__ list,
    const int32_t* __restrict__ count, const TileSum* __restrict__ info, int32_t n_qt,
    int32_t L_pad, int32_t n_work, PfCached cc) {
  prefill_attn_body<uint16_t, D, CACHED>(q, k, v, o, H, L, qs, kvs, os, c2, vu, L_meta, list,
                                         count, info, n_qt, L_pad, n_work, cc);
}

template <int D, bool CACHED>
__global__ __launch_bounds__(PF_THREADS) void prefill_attn_kernel_f32(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    float* __restrict__ o, int32_t H, int32_t L, int64_t qs, int64_t kvs, int64_t os, float c2,
    const int32_t* __restrict__ vu, int32_t L_meta, const uint32_t* __restrict__ list,
    const int32_t* __restrict__ count, const TileSum* __restrict__ info, int32_t n_qt,
    int32_t L_pad, int32_t n_work, PfCached cc) {
  prefill_attn_body<float, D, CACHED>(q, k, v, o, H, L, qs, kvs, os, c2, vu, L_meta, list, count,
                                      info, n_qt, L_pad, n_work, cc);
}

template <typename T, int D, bool CACHED>
static int launch_prefill(const void* q, const void* k, const void* v, void* o, int32_t b,
                          int32_t H, int32_t L, int64_t qs, int64_t kvs, int64_t os, float scale,
                          const int32_t* vu, int32_t L_meta, uint32_t* list, int32_t* count,
                          TileSum* info, int32_t n_qt, int32_t L_pad, PfCached cc, bool plan,
                          hipStream_t stream) {
  if (plan) {
    prefill_plan_kernel<CACHED><<<dim3(n_qt, b), 256, 0, stream>>>(vu, L_meta, L, n_qt, L_pad,
                                                                   list, count, info, cc);
    int rc = hip_check(hipGetLastError(), "span_masked_prefill_attn: plan launch");
    if (rc) return rc;
  }
  const int n_work = b * H * n_qt;
  if constexpr (sizeof(T) == 2)
    prefill_attn_kernel_bf16<D, CACHED><<<n_work, PF_THREADS, 0, stream>>>(
        static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
        static_cast<T*>(o), H, L, qs, kvs, os, scale * PF_LOG2E, vu, L_meta, list, count, info,
        n_qt, L_pad, n_work, cc);
  else
    prefill_attn_kernel_f32<D, CACHED><<<n_work, PF_THREADS, 0, stream>>>(
        static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v),
        static_cast<T*>(o), H, L, qs, kvs, os, scale * PF_LOG2E, vu, L_meta, list, count, info,
        n_qt, L_pad, n_work, cc);
  return hip_check(hipGetLastError(), "span_masked_prefill_attn: launch");
}

template <bool CACHED>
static int dispatch_prefill(const void* q, const void* k, const void* v, void* o, int32_t b,
                            int32_t H, int32_t L, int32_t d_head, sckv_dtype dt, int64_t qs,
                            int64_t kvs, int64_t os, float scale, const int32_t* vu,
                            int32_t L_meta, uint32_t* list, int32_t* cnt, TileSum* info,
                            int32_t n_qt, int32_t L_pad, PfCached cc, bool plan,
                            hipStream_t stream) {
  if (dt == SCKV_BF16)
    return d_head == 64 ? launch_prefill<uint16_t, 64, CACHED>(q, k, v, o, b, H, L, qs, kvs, os, scale, vu, L_meta, list, cnt, info, n_qt, L_pad, cc, plan, stream)
                        : launch_prefill<uint16_t, 80, CACHED>(q, k, v, o, b, H, L, qs, kvs, os, scale, vu, L_meta, list, cnt, info, n_qt, L_pad, cc, plan, stream);
  return d_head == 64 ? launch_prefill<float, 64, CACHED>(q, k, v, o, b, H, L, qs, kvs, os, scale, vu, L_meta, list, cnt, info, n_qt, L_pad, cc, plan, stream)
                      : launch_prefill<float, 80, CACHED>(q, k, v, o, b, H, L, qs, kvs, os, scale, vu, L_meta, list, cnt, info, n_qt, L_pad, cc, plan, stream);
}

static void plan_geometry(int32_t L, int32_t* n_qt, int32_t* L_pad) {
  *n_qt = (L + PF_BQ - 1) / PF_BQ;
  *L_pad = *n_qt * PF_BQ;
}

// cached: a query block lists at most row0 + nq <= L_cap rows
static void plan_geometry_cached(int32_t nq, int32_t L_cap, int32_t* n_qt, int32_t* L_pad) {
  *n_qt = (nq + PF_BQ - 1) / PF_BQ;
  *L_pad = (L_cap + PF_BQ - 1) / PF_BQ * PF_BQ;
}

}  // namespace sckv

using namespace sckv;

extern "C" size_t sckv_prefill_workspace_bytes(int32_t b, int32_t L) {
  if (b <= 0 || L <= 0) return 0;
  int32_t n_qt, L_pad;
  plan_geometry(L, &n_qt, &L_pad);
  const size_t list = (size_t)b * n_qt * L_pad * sizeof(uint32_t);
  const size_t sums = (size_t)b * n_qt * (L_pad / 64) * sizeof(TileSum);
  const size_t cnt = ((size_t)b * n_qt * sizeof(int32_t) + 255) / 256 * 256;
  return list + sums + cnt;
}

// workspace of the plain prefill: list entries | tile summaries | counts
struct PlainPlan {
  uint32_t* list;
  TileSum* sums;
  int32_t* cnt;
  int32_t n_qt, L_pad;
};
static PlainPlan plain_plan(void* ws, int32_t b, int32_t L) {
  PlainPlan p;
  plan_geometry(L, &p.n_qt, &p.L_pad);
  const size_t list_bytes = (size_t)b * p.n_qt * p.L_pad * sizeof(uint32_t);
  const size_t sum_bytes = (size_t)b * p.n_qt * (p.L_pad / 64) * sizeof(TileSum);
  p.list = static_cast<uint32_t*>(ws);
  p.sums = reinterpret_cast<TileSum*>(static_cast<char*>(ws) + list_bytes);
  p.cnt = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + list_bytes + sum_bytes);
  return p;
}

// checks shared by the plan-only call and the attention calls
static int check_plan_args(const char* W, const int32_t* vu, int32_t b, int32_t L, int32_t L_meta,
                           const void* ws, size_t ws_bytes) {
  if (!vu || !ws) return fail(SCKV_EINVAL, std::string(W) + ": null pointer");
  if (b <= 0 || L <= 0) return fail(SCKV_EINVAL, std::string(W) + ": sizes must be positive");
  if (L > 32768) return fail(SCKV_EUNSUP, std::string(W) + ": L above 32768");
  if (L_meta < L) return fail(SCKV_EINVAL, std::string(W) + ": L_meta < L");
  if (!aligned16(ws)) return fail(SCKV_EINVAL, std::string(W) + ": workspace must be 16-byte aligned");
  if (ws_bytes < sckv_prefill_workspace_bytes(b, L))
    return fail(SCKV_EINVAL, std::string(W) + ": workspace too small");
  return SCKV_OK;
}

static int prefill_entry(const char* W, bool plan, const void* q, const void* k, const void* v,
                         void* o, int32_t b, int32_t H, int32_t L, int32_t d_head,
                         int64_t q_stride_bh, int64_t kv_stride_bh, int64_t o_stride_bh,
                         sckv_dtype dt, float scale, const int32_t* vu, int32_t L_meta, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  clear_error();
  if (!q || !k || !v || !o) return fail(SCKV_EINVAL, std::string(W) + ": null pointer");
  int rc = check_plan_args(W, vu, b, L, L_meta, ws, ws_bytes);
  if (rc) return rc;
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, std::string(W) + ": unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, std::string(W) + ": d_head must be 64 or 80");
  if (H <= 0) return fail(SCKV_EINVAL, std::string(W) + ": sizes must be positive");
  const int64_t rowlen = (int64_t)L * d_head;
  if (q_stride_bh < rowlen || kv_stride_bh < rowlen || o_stride_bh < rowlen)
    return fail(SCKV_EINVAL, std::string(W) + ": slice stride smaller than L*d_head");
  const int eb = elem_bytes(dt);
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
      (q_stride_bh * eb) % 16 || (kv_stride_bh * eb) % 16 || (o_stride_bh * eb) % 16)
    return fail(SCKV_EINVAL, std::string(W) + ": buffers and strides must be 16-byte aligned");
  if (!(scale > 0.f) || std::isinf(scale)) return fail(SCKV_EINVAL, std::string(W) + ": scale must be finite and > 0");
  const PlainPlan p = plain_plan(ws, b, L);
  if ((int64_t)b * H * p.n_qt > 0x7fffffff) return fail(SCKV_EUNSUP, std::string(W) + ": grid too large");
  return dispatch_prefill<false>(q, k, v, o, b, H, L, d_head, dt, q_stride_bh, kv_stride_bh,
                                 o_stride_bh, scale, vu, L_meta, p.list, p.cnt, p.sums, p.n_qt,
                                 p.L_pad, PfCached{}, plan, stream);
}

extern "C" int span_masked_prefill_attn(const void* q, const void* k, const void* v, void* o,
                                        int32_t b, int32_t H, int32_t L, int32_t d_head,
                                        int64_t q_stride_bh, int64_t kv_stride_bh,
                                        int64_t o_stride_bh, sckv_dtype dt, float scale,
                                        const int32_t* vu, int32_t L_meta, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  return prefill_entry("span_masked_prefill_attn", true, q, k, v, o, b, H, L, d_head, q_stride_bh,
                       kv_stride_bh, o_stride_bh, dt, scale, vu, L_meta, ws, ws_bytes, stream);
}

extern "C" int sckv_prefill_plan(const int32_t* vu, int32_t L_meta, int32_t b, int32_t L,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  const char* W = "sckv_prefill_plan";
  int rc = check_plan_args(W, vu, b, L, L_meta, ws, ws_bytes);
  if (rc) return rc;
  const PlainPlan p = plain_plan(ws, b, L);
  prefill_plan_kernel<false><<<dim3(p.n_qt, b), 256, 0, stream>>>(vu, L_meta, L, p.n_qt, p.L_pad,
                                                                  p.list, p.cnt, p.sums,
                                                                  PfCached{});
  return hip_check(hipGetLastError(), "sckv_prefill_plan: launch");
}

extern "C" int span_masked_prefill_attn_planned(const void* q, const void* k, const void* v,
                                                void* o, int32_t b, int32_t H, int32_t L,
                                                int32_t d_head, int64_t q_stride_bh,
                                                int64_t kv_stride_bh, int64_t o_stride_bh,
                                                sckv_dtype dt, float scale, const int32_t* vu,
                                                int32_t L_meta, void* ws, size_t ws_bytes,
                                                hipStream_t stream) {
  return prefill_entry("span_masked_prefill_attn_planned", false, q, k, v, o, b, H, L, d_head,
                       q_stride_bh, kv_stride_bh, o_stride_bh, dt, scale, vu, L_meta, ws,
                       ws_bytes, stream);
}

extern "C" size_t sckv_prefill_cached_workspace_bytes(int32_t b, int32_t nq, int32_t L_cap) {
  if (b <= 0 || nq <= 0 || L_cap <= 0) return 0;
  int32_t n_qt, L_pad;
  plan_geometry_cached(nq, L_cap, &n_qt, &L_pad);
  const size_t list = (size_t)b * n_qt * L_pad * sizeof(uint32_t);  // entries, then rows
  const size_t sums = (size_t)b * n_qt * (L_pad / 64) * sizeof(TileSum);
  const size_t cnt = ((size_t)b * n_qt * sizeof(int32_t) + 255) / 256 * 256;
  return 2 * list + sums + cnt;
}

// workspace of the cached prefill: list entries | their cache rows | tile
// summaries | counts
struct CachedPlan {
  uint32_t* list;
  TileSum* sums;
  int32_t* cnt;
  PfCached cc;
  int32_t n_qt, L_pad;
};
static CachedPlan cached_plan(void* ws, int32_t b, int32_t nq, int32_t L_cap, int32_t tok0,
                              const int32_t* row0, const int32_t* tok_idx, int32_t* status) {
  CachedPlan p;
  plan_geometry_cached(nq, L_cap, &p.n_qt, &p.L_pad);
  const size_t list_bytes = (size_t)b * p.n_qt * p.L_pad * sizeof(uint32_t);
  const size_t sum_bytes = (size_t)b * p.n_qt * (p.L_pad / 64) * sizeof(TileSum);
  char* base = static_cast<char*>(ws);
  p.list = reinterpret_cast<uint32_t*>(base);
  p.cc.rows = reinterpret_cast<uint32_t*>(base + list_bytes);
  p.sums = reinterpret_cast<TileSum*>(base + 2 * list_bytes);
  p.cnt = reinterpret_cast<int32_t*>(base + 2 * list_bytes + sum_bytes);
  p.cc.row0 = row0;
  p.cc.tok = tok_idx;
  p.cc.tok0 = tok0;
  p.cc.L_cap = L_cap;
  p.cc.status = status;
  return p;
}

// checks shared by the cached plan-only call and the cached attention calls
static int check_cached_plan_args(const char* W, const int32_t* vu, int32_t L_meta, int32_t tok0,
                                  const int32_t* row0, const int32_t* tok_idx, int32_t L_cap,
                                  int32_t b, int32_t nq, const void* ws, size_t ws_bytes) {
  if (!vu || !row0 || !tok_idx || !ws) return fail(SCKV_EINVAL, std::string(W) + ": null pointer");
  if (b <= 0 || nq <= 0 || L_cap <= 0)
    return fail(SCKV_EINVAL, std::string(W) + ": sizes must be positive");
  if (L_cap > 32768 || nq > L_cap) return fail(SCKV_EUNSUP, std::string(W) + ": nq <= L_cap <= 32768 required");
  // list entries hold a token in 24 bits; 0xffffff marks padding
  if (L_meta <= 0 || L_meta >= (int32_t)PF_NONE)
    return fail(SCKV_EUNSUP, std::string(W) + ": L_meta must be in (0, 2^24 - 1)");
  if (tok0 < 0 || (int64_t)tok0 + nq > L_meta)
    return fail(SCKV_EINVAL, std::string(W) + ": query tokens [tok0, tok0+nq) exceed L_meta");
  if (!aligned16(ws)) return fail(SCKV_EINVAL, std::string(W) + ": workspace must be 16-byte aligned");
  if (ws_bytes < sckv_prefill_cached_workspace_bytes(b, nq, L_cap))
    return fail(SCKV_EINVAL, std::string(W) + ": workspace too small");
  return SCKV_OK;
}

static int cached_entry(const char* W, bool plan, const void* q, const void* k_cache,
                        const void* v_cache, void* o, int32_t b, int32_t H, int32_t nq,
                        int32_t d_head, int64_t q_stride_bh, int64_t kv_stride_bh,
                        int64_t o_stride_bh, sckv_dtype dt, float scale, const int32_t* vu,
                        int32_t L_meta, int32_t tok0, const int32_t* row0, const int32_t* tok_idx,
                        int32_t L_cap, void* ws, size_t ws_bytes, int32_t* status,
                        hipStream_t stream) {
  clear_error();
  if (!q || !k_cache || !v_cache || !o) return fail(SCKV_EINVAL, std::string(W) + ": null pointer");
  int rc = check_cached_plan_args(W, vu, L_meta, tok0, row0, tok_idx, L_cap, b, nq, ws, ws_bytes);
  if (rc) return rc;
  if (!valid_dtype(dt)) return fail(SCKV_EINVAL, std::string(W) + ": unknown dtype");
  if (!supported_d(d_head)) return fail(SCKV_EUNSUP, std::string(W) + ": d_head must be 64 or 80");
  if (H <= 0) return fail(SCKV_EINVAL, std::string(W) + ": sizes must be positive");
  if (q_stride_bh < (int64_t)nq * d_head || o_stride_bh < (int64_t)nq * d_head ||
      kv_stride_bh < (int64_t)L_cap * d_head)
    return fail(SCKV_EINVAL, std::string(W) + ": slice stride too small");
  const int eb = elem_bytes(dt);
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o) ||
      (q_stride_bh * eb) % 16 || (kv_stride_bh * eb) % 16 || (o_stride_bh * eb) % 16)
    return fail(SCKV_EINVAL, std::string(W) + ": buffers and strides must be 16-byte aligned");
  if (!(scale > 0.f) || std::isinf(scale)) return fail(SCKV_EINVAL, std::string(W) + ": scale must be finite and > 0");
  const CachedPlan p = cached_plan(ws, b, nq, L_cap, tok0, row0, tok_idx, status);
  if ((int64_t)b * H * p.n_qt > 0x7fffffff) return fail(SCKV_EUNSUP, std::string(W) + ": grid too large");
  return dispatch_prefill<true>(q, k_cache, v_cache, o, b, H, nq, d_head, dt, q_stride_bh,
                                kv_stride_bh, o_stride_bh, scale, vu, L_meta, p.list, p.cnt,
                                p.sums, p.n_qt, p.L_pad, p.cc, plan, stream);
}

extern "C" int span_masked_prefill_attn_cached(
    const void* q, const void* k_cache, const void* v_cache, void* o, int32_t b, int32_t H,
    int32_t nq, int32_t d_head, int64_t q_stride_bh, int64_t kv_stride_bh, int64_t o_stride_bh,
    sckv_dtype dt, float scale, const int32_t* vu, int32_t L_meta, int32_t tok0,
    const int32_t* row0, const int32_t* tok_idx, int32_t L_cap, void* ws, size_t ws_bytes,
    int32_t* status, hipStream_t stream) {
  return cached_entry("span_masked_prefill_attn_cached", true, q, k_cache, v_cache, o, b, H, nq,
                      d_head, q_stride_bh, kv_stride_bh, o_stride_bh, dt, scale, vu, L_meta, tok0,
                      row0, tok_idx, L_cap, ws, ws_bytes, status, stream);
}

extern "C" int sckv_prefill_cached_plan(const int32_t* vu, int32_t L_meta, int32_t tok0,
                                        const int32_t* row0, const int32_t* tok_idx,
                                        int32_t L_cap, int32_t b, int32_t nq, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  clear_error();
  const char* W = "sckv_prefill_cached_plan";
  int rc = check_cached_plan_args(W, vu, L_meta, tok0, row0, tok_idx, L_cap, b, nq, ws, ws_bytes);
  if (rc) return rc;
  const CachedPlan p = cached_plan(ws, b, nq, L_cap, tok0, row0, tok_idx, nullptr);
  prefill_plan_kernel<true><<<dim3(p.n_qt, b), 256, 0, stream>>>(vu, L_meta, nq, p.n_qt, p.L_pad,
                                                                 p.list, p.cnt, p.sums, p.cc);
  return hip_check(hipGetLastError(), "sckv_prefill_cached_plan: launch");
}

extern "C" int span_masked_prefill_attn_cached_planned(
    const void* q, const void* k_cache, const void* v_cache, void* o, int32_t b, int32_t H,
    int32_t nq, int32_t d_head, int64_t q_stride_bh, int64_t kv_stride_bh, int64_t o_stride_bh,
    sckv_dtype dt, float scale, const int32_t* vu, int32_t L_meta, int32_t tok0,
    const int32_t* row0, const int32_t* tok_idx, int32_t L_cap, void* ws, size_t ws_bytes,
    int32_t* status, hipStream_t stream) {
  return cached_entry("span_masked_prefill_attn_cached_planned", false, q, k_cache, v_cache, o, b,
                      H, nq, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, dt, scale, vu,
                      L_meta, tok0, row0, tok_idx, L_cap, ws, ws_bytes, status, stream);
}
