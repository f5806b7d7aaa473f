// stream.hip -- the streaming kernels of the per-sequence sampling step (sec. 6.1, Eq. opt_sample: every
// worker runs the unchanged per-row sampling computation on its rows; the computation is the one of
// the workload of sec. 8.1: penalties, temperature, top-k, top-p, min-p, greedy, and the draw).
//
// A row of the [B, V] logits is cut into P chunks of at most CSLOTS 16-byte slots (38912 bf16 or 19456
// fp32 logits).  Six launches on the caller's stream sample a batch: the chunk kernel, the resolution
// kernel and, for the rows whose kept set has no small bound, four general-path launches (which return
// at once for every other row).
//
// The chunk kernel runs one 256-thread workgroup per chunk (four resident per CU).  A chunk workgroup
//   * issues every 16-byte load of its chunk up front with the non-temporal hint (each logit is read
//     once; the hint keeps the stream from displacing cached data), after the loads of the row's
//     token history;
//   * builds the penalty overlay of its range: the history ids that fall in the chunk go into an LDS
//     presence bitmap, a word prefix count numbers the marked positions, and their counts are
//     accumulated by number;
//   * takes the slots in arrival order: penalised elements are masked out of the registers, the rest
//     enter a running maximum and a sum of exponentials against a reference that moves with the
//     thread maximum; the penalised elements then join with their new values (LDS "extras");
//   * reduces the chunk to its max, its sum and, for rows with a top-k / min-p / top-n bound, a short
//     candidate list sorted in descending order (the bound is a provable lower limit of the chunk's
//     K-th largest value: the K-th largest per-thread maximum);
//   * writes its record and its list to the workspace with plain stores and ends.
// The resolution kernel runs one workgroup per row once the chunk kernel has finished (the end of a
// launch makes its stores visible to the next launch on the stream, whichever XCD wrote them): the
// log-sum-exp over the chunks in chunk order, top-n and the top-k threshold by ranking the list heads,
// min-p, the nucleus and the inverse-CDF draw in ascending token id on the (small) kept set.  Rows whose
// kept set has no small bound (top-p alone, no filter, lists over capacity) take the general path:
// distance histograms, the crossing bucket and the draw over re-reads of the row's logits with the
// penalty overlay rebuilt per chunk, so nothing of size [B, V] is ever written.  Such rows without a
// top-k are deferred to the general-path launches, which spread the re-reads over the row's chunks
// (k_gen_a, k_gen_b, k_gen_s) and finish each row in one workgroup (k_gen_c); rows with a top-k that
// needs the whole-row count selection are resolved by the resolution kernel itself.  No workgroup ever
// waits for another.
//
// Everything that combines values across threads, waves or chunks does so in a fixed order or in
// integers, so the results depend only on the row's values, V, the dtype and the row's alignment.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <utility>

#include "albireo.h"
#include "stream.h"

namespace {

#include "common.h"

constexpr int CT = 256;                            // threads per chunk workgroup
constexpr int CW = CT / 64;                        // waves per workgroup
constexpr int CJ = 19;                             // 16-byte register slots per thread (chunk kernel)
constexpr int GJ = 4;                              // slots per thread per re-read batch (resolution kernel)
constexpr int CSLOTS = CT * CJ;                    // body slots per chunk at most
constexpr int BMW = ((CSLOTS + 2) * 8 + 31) / 32;  // bitmap words (one bit per element, +1 slot each side)
constexpr int XCAP = ALBIREO_MAX_UNIQUE_HISTORY;   // distinct penalised positions tracked per chunk
constexpr int LCAPC = 512;                         // candidate list capacity of a chunk
constexpr int MCAP = 512;                          // kept-set capacity of the list resolution
constexpr int MAXPC = 64;                          // chunks per row
constexpr int HXN = 16;                            // plain head (threads 0-7) and tail (8-15) extras
constexpr int GEN_WORDS = 512;                     // general-path histogram area (64-bit words)
constexpr int GSTAGE = 1024;                       // 64-bit words of the resolution kernel's staging area
constexpr int HSTAGE = 4096;                       // output-history ids the resolution kernel keeps in LDS
constexpr double LN2 = 0.6931471805599453;

constexpr uint32_t PUB_FINITE = 1u << 29;  // the chunk holds a finite processed value
constexpr uint32_t PUB_OVER = 1u << 28;    // the chunk's candidate list did not fit
constexpr int REC_WORDS = 8;               // 64-bit words per chunk record (5 used)
// A row whose kept set has no small bound and no top-k is resolved chunk-parallel by three launches
// after the resolution kernel; its state between them (RS_WORDS words per row):
constexpr int RS_WORDS = 8;
constexpr uint64_t RS_DEFER = 1;  // word 0: the row is deferred
constexpr uint64_t RS_TOPP = 2;   // word 0: its kept set is a nucleus (else all values >= lo)
constexpr int SCAP = 512;         // crossing-bucket values staged per chunk
constexpr int SSTRIDE = SCAP + GEN_WORDS;  // per chunk: the staged values, then the crossing bucket's
                                           // mass per sub-bucket

// What one chunk publishes for the row's resolution (decoded form).
struct ChunkPub {
  float zmax;      // max processed value z of the chunk (+inf in rows with a bad input)
  float mref;      // reference of s (log2 units)
  float s;         // sum of 2^(z L2E - mref) over the chunk
  uint32_t flags;  // FLAG_BAD_INPUT, FLAG_LIMIT, PUB_*
  int32_t argpos;  // greedy rows: lowest position of zmax
  int32_t n_list;  // sorted candidates in the chunk's list
  float qk;        // z of list entry ceil(k / P) - 1 (-inf if the list is shorter)
  float qn;        // z of list entry ceil(n_top / P) - 1
};

struct SArgs {
  const unsigned char* logits;
  int64_t B, V, ld;
  DevParams prm;
  const float* uniforms;
  int32_t* out_ids;
  float* out_logprobs;
  int32_t n_top;
  int32_t* out_top_ids;
  float* out_top_logprobs;
  uint32_t* out_flags;
  int32_t rng_on;
  uint64_t rng_seed, rng_step;
  const int64_t* seq_ids;
  int32_t* next_tokens;
  const int32_t* backfill_dest;
  int64_t next_len;
  uint32_t seg_sps, seg_magic;  // blocked layout: slots per block, floor((2^32 - 1) / seg_sps)
  int64_t seg_gap;              // bytes between the end of a block and the start of the next
  // prompt history (repetition only) and per-sequence penalty state, in place of or beside hist_*
  const int64_t* prompt_offsets;
  const int32_t* prompt_ids;
  int64_t prompt_len;
  const int32_t* st_ids;
  const uint32_t* st_counts;
  const int32_t* st_len;
  const uint32_t* st_flags;
  int32_t st_cap;
  int32_t P;
  int32_t xcd_map;
  int64_t chunk_slots;
  int64_t grid;
  uint64_t* rec;     // [B * P * REC_WORDS] chunk records
  uint64_t* lists;   // [B * P * LCAPC] candidate keys
  uint64_t* rstate;  // [B * RS_WORDS] deferred rows' state
  uint64_t* stg;     // [B * P * SSTRIDE] deferred rows' staged crossing-bucket values and sub-buckets
  int32_t* dq;       // [2 + B] deferred rows: their count, k_gen_c's arrivals, the row indices
};

struct SRow {
  int64_t row;
  const unsigned char* rowp;
  int V, head, tail_lo, c, P;
  int64_t body_slots, s0, s1;
  bool greedy, kon, minp_on, topp_on, pen_on;
  float r, p, minp, rep, freq, pres;
  int k;
  int64_t h_lo, h_hi;  // output history [h_lo, h_hi)
  int64_t p_lo, p_hi;  // prompt history
  int st_n;            // penalty state entries
  uint32_t flags;
};

// Penalty overlay of one chunk in LDS.
struct PenLds {
  uint32_t bitmap[BMW];      // presence of the chunk's positions in the row's history
  uint16_t wpref[BMW + 2];   // set bits in the bitmap words before each word
  uint32_t xval[XCAP];       // per penalised position: its count, then its new value
  uint32_t xorig[XCAP];      // chunk kernel: per penalised position, its logit as loaded
};

// LDS of one workgroup: the chunk phase, the general path and the list resolution share the bytes.
struct SSm {
  union {
    struct {
      PenLds p;
      uint64_t list[LCAPC];      // candidate keys; the general path's staged crossing bucket
      uint64_t gen[GEN_WORDS];   // general path: histograms
    } c;
    uint64_t key[(sizeof(PenLds) + 8 * (LCAPC + GEN_WORDS)) / 8];  // list resolution staging
  };
  ChunkPub pub[MAXPC];
  uint64_t cm[MAXPC];  // general path: per-chunk kept masses
  int32_t cnt[MAXPC];
  int32_t cut[MAXPC];
  int32_t hx_pos[HXN];
  float hx_val[HXN];
  float wred[3][CW];
  uint64_t qred[CW];
  int32_t n_list;
  int32_t hst_on;      // resolution kernel: the row's output history is in r_hstage, grouped by chunk
  int32_t hoff[MAXPC + 1];  // resolution kernel: chunk c's history ids are r_hstage[hoff[c], hoff[c + 1])
  int32_t hcur[MAXPC];      // resolution kernel: scatter cursors of that grouping
  uint32_t flags;
  int32_t ov_red[CW];  // the overlay build's block scan (callers keep counters in bc_i across it)
  int32_t bc_i[4];
  float bc_f[4];
  uint64_t bc_q[2];
  int32_t top_id[ALBIREO_MAX_TOP_N];
  float top_lp[ALBIREO_MAX_TOP_N];
};
constexpr int MSTAGE = (int)(sizeof(SSm::key) / 8);
static_assert(MSTAGE >= 2048, "list staging area below 2048 keys");
static_assert(sizeof(SSm) <= 40 * 1024, "LDS of a chunk workgroup exceeds a quarter of a gfx950 CU");

// The resolution kernel's LDS beside SSm, at namespace scope so that every access to it compiles to an
// LDS instruction (a pointer kept in SSm is generic, and generic accesses wait on the memory counters
// too): the general path's staging area and the row's output history.  Only the resolution kernel
// refers to them, so only it allocates them.
__shared__ uint64_t r_gstage[GSTAGE];
__shared__ int32_t r_hstage[HSTAGE];

// Hide the register slots' contents from the optimiser between passes, so that it unpacks the slots
// again in every pass instead of keeping all unpacked (or scaled) values of the previous one alive.
template <int N>
__device__ __forceinline__ void reload_barrier(uint4 (&d)[N]) {
  static_for<N>([&](auto J) {
    constexpr int j = decltype(J)::value;
    uint32_t x = d[j].x, y = d[j].y, z = d[j].z, w = d[j].w;
    asm volatile("" : "+v"(x), "+v"(y), "+v"(z), "+v"(w));
    d[j] = make_uint4(x, y, z, w);
  });
}

// Element e of a 16-byte slot, the slot taken by value (so that a run-time e selects among register
// values and never turns the register slots into addressable memory).
template <class DT>
__device__ __forceinline__ float elem(uint4 d, int e) {
  if constexpr (DT::VEC == 8) {
    const int h = e >> 1;
    uint32_t w = d.x;
    w = h == 1 ? d.y : w;
    w = h == 2 ? d.z : w;
    w = h == 3 ? d.w : w;
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  } else {
    uint32_t w = d.x;
    w = e == 1 ? d.y : w;
    w = e == 2 ? d.z : w;
    w = e == 3 ? d.w : w;
    return __uint_as_float(w);
  }
}

// ----------------------------------------------------------------------------------------------
// Workgroup reductions (4 waves; fixed combination order)
// ----------------------------------------------------------------------------------------------
__device__ __forceinline__ int blk_min_i(int v, SSm& s) {
  v = wave_min_i(v);
  __syncthreads();
  if (lane_id() == 0) s.bc_i[wave_id()] = v;
  __syncthreads();
  return min(min(s.bc_i[0], s.bc_i[1]), min(s.bc_i[2], s.bc_i[3]));
}
__device__ __forceinline__ int blk_max_i(int v, SSm& s) {
  v = wave_max_i(v);
  __syncthreads();
  if (lane_id() == 0) s.bc_i[wave_id()] = v;
  __syncthreads();
  return max(max(s.bc_i[0], s.bc_i[1]), max(s.bc_i[2], s.bc_i[3]));
}
__device__ __forceinline__ uint32_t blk_or(uint32_t v, SSm& s) {
  v = wave_or(v);
  __syncthreads();
  if (lane_id() == 0) s.bc_i[wave_id()] = (int)v;
  __syncthreads();
  return (uint32_t)(s.bc_i[0] | s.bc_i[1] | s.bc_i[2] | s.bc_i[3]);
}
__device__ __forceinline__ uint64_t blk_sum_u64(uint64_t v, SSm& s) {
  v = wave_sum_u64(v);
  __syncthreads();
  if (lane_id() == 0) s.qred[wave_id()] = v;
  __syncthreads();
  return s.qred[0] + s.qred[1] + s.qred[2] + s.qred[3];
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = ((uint64_t)(uint32_t)__shfl_xor((int)(v >> 32), o) << 32) | (uint32_t)__shfl_xor((int)v, o);
    v = w > v ? w : v;
  }
  return v;
}
__device__ __forceinline__ uint64_t blk_max_u64(uint64_t v, SSm& s) {
  v = wave_max_u64(v);
  __syncthreads();
  if (lane_id() == 0) s.qred[wave_id()] = v;
  __syncthreads();
  uint64_t r = s.qred[0];
  for (int w = 1; w < CW; ++w) r = s.qred[w] > r ? s.qred[w] : r;
  return r;
}
// exclusive prefix of v over the threads in thread order; *total = sum over all threads
__device__ __forceinline__ int blk_excl_scan_i(int v, SSm& s, int* total) {
  const int incl = wave_incl_scan_i(v);
  __syncthreads();
  if (lane_id() == 63) s.bc_i[wave_id()] = incl;
  __syncthreads();
  int off = 0;
  for (int w = 0; w < wave_id(); ++w) off += s.bc_i[w];
  *total = s.bc_i[0] + s.bc_i[1] + s.bc_i[2] + s.bc_i[3];
  return off + incl - v;
}
__device__ __forceinline__ uint64_t blk_excl_scan_u64(uint64_t v, SSm& s, uint64_t* total) {
  // inclusive scan in lane order on DPP, 64-bit
  uint64_t incl = v;
  incl += dpp_mov64<DPP_ROW_SHR + 1>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 2>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 4>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 8>(incl);
  incl += dpp_mov64<DPP_ROW_BCAST15, 0xa>(incl);
  incl += dpp_mov64<DPP_ROW_BCAST31, 0xc>(incl);
  __syncthreads();
  if (lane_id() == 63) s.qred[wave_id()] = incl;
  __syncthreads();
  uint64_t off = 0;
  for (int w = 0; w < wave_id(); ++w) off += s.qred[w];
  *total = s.qred[0] + s.qred[1] + s.qred[2] + s.qred[3];
  return off + incl - v;
}

// (mref, s) pairs: s is relative to 2^mref
__device__ __forceinline__ void lse_add(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  s = s * rel2(m, M) + s2 * rel2(m2, M);
  m = M;
}

// fixed-point mass of a kept value: 2^((z - m) L2E) in units of 2^-32
__device__ __forceinline__ uint64_t mass_of(float z, float m) {
  const float w = __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(z, m), L2E));
  return (uint64_t)((double)w * FIX_SCALE);
}

// ----------------------------------------------------------------------------------------------
// Chunk records: five 64-bit words (a 32-bit field and a float each)
// ----------------------------------------------------------------------------------------------
__device__ __forceinline__ uint64_t rec_word(uint32_t hi, float lo) {
  return ((uint64_t)hi << 32) | __float_as_uint(lo);
}
__device__ __forceinline__ void rec_store(uint64_t* g, const ChunkPub& p) {
  g[0] = rec_word(p.flags, p.zmax);
  g[1] = rec_word((uint32_t)(p.argpos + 1), p.mref);
  g[2] = rec_word((uint32_t)p.n_list, p.s);
  g[3] = rec_word(0u, p.qk);
  g[4] = rec_word(0u, p.qn);
}
__device__ __forceinline__ ChunkPub rec_load(const uint64_t* g) {
  uint64_t w[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) w[i] = g[i];
  ChunkPub p;
  p.flags = (uint32_t)(w[0] >> 32);
  p.zmax = __uint_as_float((uint32_t)w[0]);
  p.argpos = (int32_t)(uint32_t)(w[1] >> 32) - 1;
  p.mref = __uint_as_float((uint32_t)w[1]);
  p.n_list = (int32_t)(uint32_t)(w[2] >> 32);
  p.s = __uint_as_float((uint32_t)w[2]);
  p.qk = __uint_as_float((uint32_t)w[3]);
  p.qn = __uint_as_float((uint32_t)w[4]);
  return p;
}

// ----------------------------------------------------------------------------------------------
// Row geometry and parameters
// ----------------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t seg_block(const SArgs& a, uint32_t q) {
  uint32_t g = __umulhi(q, a.seg_magic);
  if (q - g * a.seg_sps >= a.seg_sps) ++g;
  return g;
}
template <class DT, bool SEG>
__device__ __forceinline__ const uint4* slot_ptr(const SArgs& a, const SRow& R, int64_t slot) {
  int64_t off = ((int64_t)R.head + slot * DT::VEC) * DT::ES;
  if constexpr (SEG) off += (int64_t)seg_block(a, (uint32_t)slot) * a.seg_gap;
  return reinterpret_cast<const uint4*>(R.rowp + off);
}
template <class DT, bool SEG>
__device__ __forceinline__ float load_elem(const SArgs& a, const SRow& R, int64_t pos) {
  int64_t off = pos * DT::ES;
  if constexpr (SEG) off += (int64_t)seg_block(a, (uint32_t)(pos / DT::VEC)) * a.seg_gap;
  return DT::load1(R.rowp + off, 0);
}

template <class DT, bool SEG>
__device__ __forceinline__ void row_setup(const SArgs& a, int64_t row, int c, SRow& R) {
  R.row = row;
  R.c = c;
  R.P = a.P;
  R.V = (int)a.V;
  R.rowp = a.logits + row * a.ld * DT::ES;
  int head = 0;
  if constexpr (!SEG) {
    const uint64_t addr = reinterpret_cast<uint64_t>(R.rowp);
    head = (int)(((16u - (uint32_t)(addr & 15u)) & 15u) / DT::ES);
    if (head > R.V) head = R.V;
  }
  R.head = head;
  R.body_slots = (R.V - head) / DT::VEC;
  R.tail_lo = head + (int)R.body_slots * DT::VEC;
  R.s0 = (int64_t)c * a.chunk_slots;
  if (R.s0 > R.body_slots) R.s0 = R.body_slots;
  R.s1 = R.s0 + a.chunk_slots;
  if (R.s1 > R.body_slots) R.s1 = R.body_slots;

  const DevParams& q = a.prm;
  float T = sload(q.temperature ? q.temperature + row : &kParamDefaults[0]);
  float p = sload(q.top_p ? q.top_p + row : &kParamDefaults[1]);
  float mp = sload(q.min_p ? q.min_p + row : &kParamDefaults[2]);
  float rep = sload(q.rep ? q.rep + row : &kParamDefaults[3]);
  float freq = sload(q.freq ? q.freq + row : &kParamDefaults[4]);
  float pres = sload(q.pres ? q.pres + row : &kParamDefaults[5]);
  const int k = sload(q.top_k ? q.top_k + row : &kZeroI32[0]);
  const int64_t* ho = q.hist_offsets ? q.hist_offsets + row : &kZeroI64[0];
  const int64_t lo = sload(ho), hi = sload(ho + 1);
  uint32_t flags = 0;
  if (!isfinite(T)) { flags |= FLAG_BAD_PARAM; T = 1.0f; }
  if (isnan(p)) { flags |= FLAG_BAD_PARAM; p = 1.0f; }
  if (isnan(mp)) { flags |= FLAG_BAD_PARAM; mp = 0.0f; }
  if (!(rep > 0.0f) || isinf(rep)) { flags |= FLAG_BAD_PARAM; rep = 1.0f; }
  if (!isfinite(freq)) { flags |= FLAG_BAD_PARAM; freq = 0.0f; }
  if (!isfinite(pres)) { flags |= FLAG_BAD_PARAM; pres = 0.0f; }
  R.greedy = T < 1e-5f;
  if (R.greedy) flags |= FLAG_GREEDY;
  R.r = R.greedy ? 1.0f : (float)(1.0 / (double)T);
  R.k = k;
  R.kon = !R.greedy && k > 0 && (int64_t)k < a.V;
  R.minp_on = !R.greedy && mp > 0.0f;
  R.minp = mp > 1.0f ? 1.0f : mp;
  R.topp_on = !R.greedy && p < 1.0f;
  R.p = p;
  R.rep = rep;
  R.freq = freq;
  R.pres = pres;
  R.pen_on = false;
  R.h_lo = R.h_hi = 0;
  R.p_lo = R.p_hi = 0;
  R.st_n = 0;
  if (q.hist_offsets) {
    if (lo < 0 || hi < lo || hi > q.hist_len) {
      flags |= FLAG_BAD_PARAM;
    } else if (hi > lo) {
      R.pen_on = true;
      R.h_lo = lo;
      R.h_hi = hi;
    }
  }
  if (a.prompt_offsets) {
    const int64_t plo = sload(a.prompt_offsets + row), phi = sload(a.prompt_offsets + row + 1);
    if (plo < 0 || phi < plo || phi > a.prompt_len) {
      flags |= FLAG_BAD_PARAM;
    } else if (phi > plo) {
      R.pen_on = true;
      R.p_lo = plo;
      R.p_hi = phi;
    }
  }
  if (a.st_len) {
    const int n = sload(a.st_len + row);
    R.st_n = n < 0 ? 0 : (n > a.st_cap ? a.st_cap : n);
    if (R.st_n > 0) R.pen_on = true;
  }
  R.flags = flags;
}

// body slots [s0, s1) of chunk c
__device__ __forceinline__ void chunk_range(const SArgs& a, const SRow& R, int c, int64_t& s0, int64_t& s1) {
  s0 = (int64_t)c * a.chunk_slots;
  if (s0 > R.body_slots) s0 = R.body_slots;
  s1 = s0 + a.chunk_slots;
  if (s1 > R.body_slots) s1 = R.body_slots;
}
// first and one-past-last row position of chunk c
__device__ __forceinline__ int chunk_lo(const SArgs& a, const SRow& R, int c, int vec) {
  if (c == 0) return 0;
  int64_t s = (int64_t)c * a.chunk_slots;
  if (s > R.body_slots) s = R.body_slots;
  return R.head + (int)s * vec;
}
__device__ __forceinline__ int chunk_hi(const SArgs& a, const SRow& R, int c, int vec) {
  if (c == R.P - 1) return R.V;
  int64_t s = (int64_t)(c + 1) * a.chunk_slots;
  if (s > R.body_slots) s = R.body_slots;
  return R.head + (int)s * vec;
}
__device__ __forceinline__ int chunk_of(const SArgs& a, const SRow& R, int vec, int pos) {
  int c = 0;
  while (c < R.P - 1 && pos >= chunk_hi(a, R, c, vec)) ++c;
  return c;
}

// Row position of the penalised extras entry of rank i (the i-th set bit of the bitmap).
__device__ __forceinline__ int pos_of_rank(const SSm& s, int nwords, int64_t e_base, int i) {
  int lo = 0, hi = nwords - 1;
  while (lo < hi) {  // last word whose prefix count is <= i
    const int mid = (lo + hi + 1) >> 1;
    if ((int)s.c.p.wpref[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  uint32_t w = s.c.p.bitmap[lo];
  for (int q = i - (int)s.c.p.wpref[lo]; q > 0; --q) w &= w - 1;
  return (int)(e_base + lo * 32 + __builtin_ctz(w));
}

// ----------------------------------------------------------------------------------------------
// The penalty overlay of chunk c (body slots [s0, s1)): bit b of the bitmap stands for row position
// e_base + b with e_base = head + (s0 - 1) VEC, so the slot before and the slot after the chunk (the
// unaligned head of chunk 0, the tail of the last chunk) have bits too.  Every history id in the
// chunk's positions marks its bit; word prefix counts number the marked positions; per number, the
// output count (bits 0-30) and the prompt mark (bit 31).  The first HPT * CT history ids come from the
// caller's registers (hreg, this thread's share), the rest from memory.  Returns the number of tracked
// positions (at most XCAP; past that the highest positions are left out and FLAG_LIMIT is set) and ORs
// FLAG_BAD_INPUT / FLAG_LIMIT into *fl.
// ----------------------------------------------------------------------------------------------
template <int HPT>
__device__ __forceinline__ int build_overlay(const SArgs& a, const SRow& R, SSm& s, int c, int64_t s0, int64_t s1,
                                             int vec, const int32_t (&hreg)[HPT > 0 ? HPT : 1], uint32_t* fl) {
  const int t = threadIdx.x;
  const int64_t e_base = (int64_t)R.head + (s0 - 1) * vec;
  const int nwords = (int)(((s1 - s0 + 2) * vec + 31) >> 5);
  for (int w = t; w < nwords; w += CT) s.c.p.bitmap[w] = 0;
  __syncthreads();
  const int64_t e_lo = c == 0 ? 0 : (int64_t)R.head + s0 * vec;
  const int64_t e_hi = c == R.P - 1 ? (int64_t)R.V : (int64_t)R.head + s1 * vec;
  uint32_t bad = 0;
  // ids [lo, hi) of an array, IDU loads per thread in flight before any is used (unconditional: an
  // index past the range reloads the first of the group); f(id, index)
  constexpr int IDU = 4;
  auto for_ids = [&](const int32_t* ids, int64_t lo, int64_t hi, auto&& f) __attribute__((always_inline)) {
    for (int64_t h0 = lo + t; h0 < hi; h0 += IDU * (int64_t)CT) {
      int32_t v[IDU];
#pragma unroll
      for (int q = 0; q < IDU; ++q) {
        const int64_t h = h0 + (int64_t)q * CT;
        v[q] = ids[h < hi ? h : h0];
      }
#pragma unroll
      for (int q = 0; q < IDU; ++q) {
        const int64_t h = h0 + (int64_t)q * CT;
        if (h < hi) f(v[q], h);
      }
    }
  };
  auto mark = [&](int32_t id) {
    if (id < 0 || id >= R.V) {
      bad = 1;
    } else if (id >= e_lo && id < e_hi) {
      const int b = (int)(id - e_base);
      atomicOr(&s.c.p.bitmap[b >> 5], 1u << (b & 31));
    }
  };
  // the output history: the first HPT * CT ids from the caller's registers and the rest from memory,
  // or (resolution kernel, HPT = 0) all of it from its LDS copy, indexed from 0
  const int64_t h_reg_end = min(R.h_hi, R.h_lo + (int64_t)HPT * CT);  // ids held in hreg
  auto for_hist = [&](auto&& f) __attribute__((always_inline)) {
    if constexpr (HPT == 0) {
      if (s.hst_on) {  // only this chunk's ids (the others could not mark or count anything here)
        for_ids(r_hstage, s.hoff[c], s.hoff[c + 1], f);
        return;
      }
    }
    for_ids(a.prm.hist_ids, h_reg_end, R.h_hi, f);
  };
  static_for<HPT>([&](auto Q) {
    constexpr int q = decltype(Q)::value;
    if (R.h_lo + t + (int64_t)q * CT < h_reg_end) mark(hreg[q]);
  });
  for_hist([&](int32_t id, int64_t) { mark(id); });
  for_ids(a.prompt_ids, R.p_lo, R.p_hi, [&](int32_t id, int64_t) { mark(id); });
  const int32_t* st_row = a.st_ids + R.row * a.st_cap;
  for_ids(st_row, 0, R.st_n, [&](int32_t id, int64_t) { mark(id); });
  if (bad) *fl |= FLAG_BAD_INPUT;
  __syncthreads();
  const int wpt = (nwords + CT - 1) / CT;
  const int w0 = t * wpt;
  int loc = 0;
  for (int q = 0; q < wpt; ++q)
    if (w0 + q < nwords) loc += __popc(s.c.p.bitmap[w0 + q]);
  int tot;
  int ex;
  {  // exclusive scan of loc in thread order through ov_red (bc_i belongs to the callers)
    const int incl = wave_incl_scan_i(loc);
    if (lane_id() == 63) s.ov_red[wave_id()] = incl;
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave_id(); ++w) off += s.ov_red[w];
    tot = s.ov_red[0] + s.ov_red[1] + s.ov_red[2] + s.ov_red[3];
    ex = off + incl - loc;
  }
  for (int q = 0; q < wpt; ++q)
    if (w0 + q < nwords) {
      s.c.p.wpref[w0 + q] = (uint16_t)min(ex, 0xffff);
      ex += __popc(s.c.p.bitmap[w0 + q]);
    }
  const int n_x = tot < XCAP ? tot : XCAP;
  if (tot > XCAP) *fl |= FLAG_LIMIT;
  for (int i = t; i < n_x; i += CT) s.c.p.xval[i] = 0;
  __syncthreads();
  // per numbered position: the output count in bits 0-30, the prompt mark in bit 31
  auto count = [&](int32_t id, uint32_t add, uint32_t mark_bits) {
    if (id >= e_lo && id < e_hi) {
      const int b = (int)(id - e_base);
      const int w = b >> 5;
      const int rank = (int)s.c.p.wpref[w] + __popc(s.c.p.bitmap[w] & ((1u << (b & 31)) - 1u));
      if (rank < XCAP) {
        if (add) atomicAdd(&s.c.p.xval[rank], add);
        if (mark_bits) atomicOr(&s.c.p.xval[rank], mark_bits);
      }
    }
  };
  static_for<HPT>([&](auto Q) {
    constexpr int q = decltype(Q)::value;
    if (R.h_lo + t + (int64_t)q * CT < h_reg_end) count(hreg[q], 1u, 0u);
  });
  for_hist([&](int32_t id, int64_t) { count(id, 1u, 0u); });
  for_ids(a.prompt_ids, R.p_lo, R.p_hi, [&](int32_t id, int64_t) { count(id, 0u, 0x80000000u); });
  const int32_t* st_cnt = reinterpret_cast<const int32_t*>(a.st_counts + R.row * a.st_cap);
  for_ids(st_cnt, 0, R.st_n, [&](int32_t cvi, int64_t e) {
    const uint32_t cv = (uint32_t)cvi;
    count(st_row[e], cv & 0x7fffffffu, cv & 0x80000000u);
  });
  __syncthreads();
  return n_x;
}

// rank of the marked bit b of the overlay, or -1 when b is not marked or not tracked
__device__ __forceinline__ int overlay_rank(const SSm& s, int b) {
  const int w = b >> 5;
  const uint32_t bw = s.c.p.bitmap[w];
  if (!((bw >> (b & 31)) & 1u)) return -1;
  const int rank = (int)s.c.p.wpref[w] + __popc(bw & ((1u << (b & 31)) - 1u));
  return rank < XCAP ? rank : -1;
}

// ----------------------------------------------------------------------------------------------
// Re-reading a chunk (general path of the resolving workgroup): f(z, pos) for every processed value of
// chunk c -- penalties from a rebuilt overlay, canonical z -- in no particular order.  A penalised
// position is visited twice, first as -inf (masked in the slot loop, which then needs no per-element
// branch) and then with its new value, so every f must ignore -inf.  Every thread of the workgroup must
// call it (it synchronises).
// ----------------------------------------------------------------------------------------------
// hreg: the caller's register copy of the row's first HPT * CT history ids (this thread's share), read
// by the overlay build instead of memory.
template <class DT, bool SEG, int HPT, class F>
__device__ __forceinline__ void for_chunk_h(const SArgs& a, const SRow& R, SSm& s, int c,
                                            const int32_t (&hreg)[HPT > 0 ? HPT : 1], F&& f) {
  constexpr int VEC = DT::VEC;
  const int t = threadIdx.x;
  int64_t s0, s1;
  chunk_range(a, R, c, s0, s1);
  const int ns = (int)(s1 - s0);
  int hpos = -1;
  if (c == 0 && t < R.head) hpos = t;
  else if (c == R.P - 1 && t >= 8 && t < 8 + (R.V - R.tail_lo)) hpos = R.tail_lo + (t - 8);
  const float hx = hpos >= 0 ? load_elem<DT, SEG>(a, R, hpos) : 0.0f;
  const int64_t e_base = (int64_t)R.head + (s0 - 1) * VEC;
  int n_x = 0;
  bool x_all = true;  // every marked position is tracked: the element loop masks them all
  if (R.pen_on) {
    uint32_t fl = 0;
    n_x = build_overlay<HPT>(a, R, s, c, s0, s1, VEC, hreg, &fl);
    x_all = !(fl & FLAG_LIMIT);
  }
  const float r = R.r;
  auto value = [&](float x, int pos) __attribute__((always_inline)) -> float {
    if (R.pen_on) {
      const int rk = overlay_rank(s, (int)(pos - e_base));
      if (rk >= 0) x = penalise_cv(x, s.c.p.xval[rk], R.rep, R.freq, R.pres);
    }
    return canon(x, r);
  };
  // batches of CT * GJ slots, slot j * CT + t of a batch to thread t; every load of a batch is issued
  // before any is used (indices clamped into the batch)
  for (int b0 = 0; b0 < ns; b0 += CT * GJ) {
    const int nb = min(ns - b0, CT * GJ);
    uint4 d[GJ];
    static_for<GJ>([&](auto J) {
      constexpr int j = decltype(J)::value;
      d[j] = *slot_ptr<DT, SEG>(a, R, s0 + b0 + min(j * CT + t, nb - 1));
    });
    static_for<GJ>([&](auto J) {
      constexpr int j = decltype(J)::value;
      if (j * CT + t < nb) {
        const int l = b0 + j * CT + t;  // the slot within the chunk
        const int p0 = R.head + (int)(s0 + l) * VEC;
        // the slot's overlay bits, one LDS word per slot (a slot's bits share one word)
        uint32_t word = 0, bits = 0, wpre = 0;
        const int ob = (l + 1) * VEC;
        if (R.pen_on) {
          word = s.c.p.bitmap[ob >> 5];
          bits = (word >> (ob & 31)) & ((1u << VEC) - 1u);
        }
        if (x_all) {
          // marked values are visited below with their new values; here they are -inf (ignored)
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const float x = ((bits >> e) & 1u) ? -INFINITY : elem<DT>(d[j], e);
            f(canon(x, r), p0 + e);
          }
        } else {
          if (bits) wpre = s.c.p.wpref[ob >> 5];
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            float x = elem<DT>(d[j], e);
            if ((bits >> e) & 1u) {
              const int rk = (int)wpre + __popc(word & ((1u << ((ob & 31) + e)) - 1u));
              if (rk < XCAP) x = penalise_cv(x, s.c.p.xval[rk], R.rep, R.freq, R.pres);
            }
            f(canon(x, r), p0 + e);
          }
        }
      }
    });
  }
  if (x_all && n_x > 0) {
    // the marked body positions with their new values (head and tail positions are visited above)
    const int nwords = (int)(((s1 - s0 + 2) * VEC + 31) >> 5);
    for (int i = t; i < n_x; i += CT) {
      const int pos = pos_of_rank(s, nwords, e_base, i);
      const int b = (int)(pos - e_base);
      if (b >= VEC && b < (int)(s1 - s0 + 1) * VEC)
        f(canon(penalise_cv(load_elem<DT, SEG>(a, R, pos), s.c.p.xval[i], R.rep, R.freq, R.pres), r), pos);
    }
  }
  if (hpos >= 0) f(value(hx, hpos), hpos);
  __syncthreads();  // the overlay is rebuilt for the next chunk
}
template <class DT, bool SEG, class F>
__device__ __forceinline__ void for_chunk(const SArgs& a, const SRow& R, SSm& s, int c, F&& f) {
  const int32_t none[1] = {0};
  for_chunk_h<DT, SEG, 0>(a, R, s, c, none, f);
}
// The first HPT * CT ids of the row's output history into registers (this thread's share, all loads in
// flight together; a dummy address when there is nothing to read), for for_chunk_h.
template <int HPT>
__device__ __forceinline__ void history_regs(const SArgs& a, const SRow& R, int32_t (&hreg)[HPT]) {
  const int t = threadIdx.x;
  const int nh = R.pen_on ? (int)min(R.h_hi - R.h_lo, (int64_t)HPT * CT) : 0;
  const int32_t* hrow = nh > 0 ? a.prm.hist_ids + R.h_lo : reinterpret_cast<const int32_t*>(a.rec);
  static_for<HPT>([&](auto Q) {
    constexpr int q = decltype(Q)::value;
    hreg[q] = hrow[min(t + q * CT, max(nh - 1, 0))];
  });
}

// ----------------------------------------------------------------------------------------------
// Resolution of a row by its last chunk workgroup
// ----------------------------------------------------------------------------------------------
// Entries of the chunk lists that the resolving workgroup loads together with the chunk records (one
// round trip): entries [0, E) of every chunk's list, SPQ per thread.  Entries past a list's end (its
// length comes with the records) are ignored.
constexpr int SPQ = 8;
struct Spec {
  uint64_t v[SPQ];
  int E;
  bool on;
};

// Stage into s.key the list entries i < imax of every chunk with z >= zthr, from the speculative
// registers (sp.on) or from the lists themselves.  The order is arbitrary (ranks are counted).  With
// cut_test, for the check of ties cut off at imax, s.cut[c] gets 1 (and s.cnt[c] the value's bits of
// chunk c's entry imax, the first one left out) when the list goes on past imax.  Returns the count,
// or -1 above cap.
__device__ __forceinline__ int stage_entries(const SArgs& a, const SRow& R, SSm& s, const Spec& sp, float zthr,
                                             int imax, int cap, bool cut_test) {
  const int P = R.P, t = threadIdx.x;
  if (t == 0) s.bc_i[2] = 0;
  if (t < P) s.cut[t] = 0;
  __syncthreads();
  const uint64_t* base = a.lists + (R.row * P) * (int64_t)LCAPC;
  auto take = [&](uint64_t key, int c, int i) {
    if (i < imax && i < s.pub[c].n_list) {
      if (cand_z(key) >= zthr) {
        const int idx = atomicAdd(&s.bc_i[2], 1);
        if (idx < cap) s.key[idx] = key;
      }
    } else if (i == imax && i < s.pub[c].n_list) {
      s.cut[c] = 1;
      s.cnt[c] = __float_as_int(cand_z(key));  // the first entry left out, for the tie test
    }
  };
  const int ilim = cut_test ? imax + 1 : imax;  // entries looked at per chunk
  if (sp.on && ilim <= sp.E) {
#pragma unroll
    for (int q = 0; q < SPQ; ++q) {
      const int f = t + q * CT;
      if (f < P * sp.E) {
        const int c = f / sp.E;
        take(sp.v[q], c, f - c * sp.E);
      }
    }
  } else {
    int emax = 0;
    for (int c = 0; c < P; ++c) emax = max(emax, min(s.pub[c].n_list, ilim));
    for (int f = t; f < P * emax; f += CT) {
      const int c = f / emax, i = f - c * emax;
      if (i < s.pub[c].n_list) take(base[(int64_t)c * LCAPC + i], c, i);
    }
  }
  __syncthreads();
  const int n = s.bc_i[2];
  __syncthreads();
  return n <= cap ? n : -1;
}

// Number of entries of arr[0, n) greater than key: one branch-free pass whose loads pipeline.
__device__ __forceinline__ int count_above(const uint64_t* arr, int n, uint64_t key) {
  int r = 0;
#pragma unroll 8
  for (int j = 0; j < n; ++j) r += arr[j] > key ? 1 : 0;
  return r;
}

// The general path visits the row's values in one of two ways: re-reads of every chunk (a pass over
// the row), or order keys staged in LDS.  Either way the visitor calls f(z) once per value.
template <class DT, bool SEG>
struct RowSrc {
  const SArgs& a;
  const SRow& R;
  SSm& s;
  template <class F>
  __device__ __forceinline__ void operator()(F&& f) const {
    for (int c = 0; c < R.P; ++c)
      for_chunk<DT, SEG>(a, R, s, c, [&](float z, int) __attribute__((always_inline)) { f(z); });
  }
};
struct StagedSrc {
  const uint32_t* keys;
  int n;
  template <class F>
  __device__ __forceinline__ void operator()(F&& f) const {
    for (int i = (int)threadIdx.x; i < n; i += CT) f(key2f(keys[i]));
  }
};
struct StagedPairs {  // (order key << 32 | position) pairs
  const uint64_t* ent;
  int n;
  template <class F>
  __device__ __forceinline__ void operator()(F&& f) const {
    for (int i = (int)threadIdx.x; i < n; i += CT) f(key2f((uint32_t)(ent[i] >> 32)));
  }
};

// General path, radix selection by count: the order key of the remaining-th largest finite value
// (counting duplicates) among those the source visits, or 0 when there are fewer.  hc: 256 LDS words.
template <class Src>
__device__ __forceinline__ uint32_t gp_kth_key(const Src& src, SSm& s, uint32_t* hc, int remaining) {
  uint32_t prefix = 0, pmask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = threadIdx.x; b < 256; b += CT) hc[b] = 0;
    __syncthreads();
    src([&](float z) __attribute__((always_inline)) {
      if (z > -INFINITY && z == z) {
        const uint32_t kk = f2key(z);
        if ((kk & pmask) == prefix) atomicAdd(&hc[(kk >> shift) & 255u], 1u);
      }
    });
    __syncthreads();
    if (threadIdx.x < 64) {
      const int l = threadIdx.x;  // lane l holds buckets 255 - 4l .. 252 - 4l (descending)
      uint32_t b4[4], sum = 0;
      for (int q = 0; q < 4; ++q) { b4[q] = hc[255 - 4 * l - q]; sum += b4[q]; }
      const uint32_t incl = wave_incl_scan_u(sum);
      const uint32_t excl = incl - sum;
      const uint64_t hit = __ballot(incl >= (uint32_t)remaining);
      if (hit == 0) {
        if (l == 0) s.bc_i[0] = -1;
      } else if (l == __builtin_ctzll(hit)) {
        uint32_t cum = excl;
        int q = 0;
        while (q < 3 && cum + b4[q] < (uint32_t)remaining) { cum += b4[q]; ++q; }
        s.bc_i[0] = 255 - 4 * l - q;
        s.bc_i[1] = remaining - (int)cum;
      }
    }
    __syncthreads();
    const int b = s.bc_i[0];
    if (b < 0) return 0u;
    remaining = s.bc_i[1];
    prefix |= (uint32_t)b << shift;
    pmask |= 255u << shift;
    __syncthreads();
  }
  return prefix;
}

// General path, radix selection by mass: the order key of the closing group among the values
// z >= tau2 that the source visits, walking them in descending order from a cumulative mass of
// `above` (the mass of every kept value above them): the first group at which the cumulative
// reaches `target`, or 0 when it never does.  hm: 256 LDS words of 64 bits.
template <class Src>
__device__ __forceinline__ uint32_t gp_topp_key(const Src& src, SSm& s, uint64_t* hm, float tau2, float m,
                                                double target, double above) {
  uint32_t prefix = 0, pmask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = threadIdx.x; b < 256; b += CT) hm[b] = 0;
    __syncthreads();
    src([&](float z) __attribute__((always_inline)) {
      if (z > -INFINITY && z >= tau2) {
        const uint32_t kk = f2key(z);
        if ((kk & pmask) == prefix)
          atomicAdd(reinterpret_cast<unsigned long long*>(&hm[(kk >> shift) & 255u]),
                    (unsigned long long)mass_of(z, m));
      }
    });
    __syncthreads();
    if (threadIdx.x < 64) {
      const int l = threadIdx.x;
      uint64_t b4[4], sum = 0;
      for (int q = 0; q < 4; ++q) { b4[q] = hm[255 - 4 * l - q]; sum += b4[q]; }
      uint64_t incl = sum;
      incl += dpp_mov64<DPP_ROW_SHR + 1>(incl);
      incl += dpp_mov64<DPP_ROW_SHR + 2>(incl);
      incl += dpp_mov64<DPP_ROW_SHR + 4>(incl);
      incl += dpp_mov64<DPP_ROW_SHR + 8>(incl);
      incl += dpp_mov64<DPP_ROW_BCAST15, 0xa>(incl);
      incl += dpp_mov64<DPP_ROW_BCAST31, 0xc>(incl);
      const uint64_t excl = incl - sum;
      const uint64_t hit = __ballot(above + (double)incl >= target);
      if (hit == 0) {
        if (l == 0) s.bc_i[0] = -1;
      } else if (l == __builtin_ctzll(hit)) {
        uint64_t cum = excl;
        int q = 0;
        while (q < 3 && above + (double)(cum + b4[q]) < target) { cum += b4[q]; ++q; }
        s.bc_i[0] = 255 - 4 * l - q;
        s.bc_q[0] = cum;
      }
    }
    __syncthreads();
    const int b = s.bc_i[0];
    if (b < 0) return 0u;
    above += (double)s.bc_q[0];
    prefix |= (uint32_t)b << shift;
    pmask |= 255u << shift;
    __syncthreads();
  }
  return prefix;
}

// First level of the general path's selections: buckets of the distance d = m - z from the row
// maximum, GD_SCALE per unit.  fl(m - z) and its product with GD_SCALE are monotone in z, so a value
// in a lower bucket is larger than every value in a higher one, and equal values share a bucket;
// masses (2^32 units) vanish from d = 32 ln 2 on, inside the last bucket.
constexpr int GDB = GEN_WORDS;
constexpr float GD_SCALE = 16.0f;
constexpr int GKCAP = 2 * GSTAGE - 256;  // crossing-bucket keys staged (u32) before a 256-word histogram
constexpr int GKCAP2 = GSTAGE;           // crossing-bucket (key, position) pairs staged

__device__ __forceinline__ int gp_dbucket(float z, float m) {
  const float d = __fmul_rn(__fsub_rn(m, z), GD_SCALE);
  return d < (float)(GDB - 1) ? (int)d : GDB - 1;
}

// One pass over the row: per distance bucket, the number (MASS false) or the fixed-point mass (MASS
// true) of the finite values z >= lo.  Then the first bucket, from the top, at which the cumulative
// reaches the target -- K for the count, p times the total for the mass -- with the cumulative of the
// buckets before it.  Returns false when the target is never reached.
template <bool MASS, class DT, bool SEG>
__device__ __forceinline__ bool gp_level1(const SArgs& a, const SRow& R, SSm& s, float lo, float m, double tgt,
                                          int& bb, uint64_t& before, uint64_t& total) {
  uint64_t* h64 = s.c.gen;
  uint32_t* h32 = reinterpret_cast<uint32_t*>(s.c.gen);
  for (int b = threadIdx.x; b < GDB; b += CT) {
    if (MASS) h64[b] = 0;
    else h32[b] = 0;
  }
  __syncthreads();
  RowSrc<DT, SEG>{a, R, s}([&](float z) __attribute__((always_inline)) {
    if (z > -INFINITY && z >= lo) {
      const int b = gp_dbucket(z, m);
      if (MASS) {
        const uint64_t w = mass_of(z, m);
        if (w) atomicAdd(reinterpret_cast<unsigned long long*>(&h64[b]), (unsigned long long)w);  // zero adds nothing
      } else {
        atomicAdd(&h32[b], 1u);
      }
    }
  });
  __syncthreads();
  constexpr int BPT = GDB / CT;  // consecutive buckets per thread
  auto hv = [&](int b) __attribute__((always_inline)) -> uint64_t { return MASS ? h64[b] : (uint64_t)h32[b]; };
  const int b0 = (int)threadIdx.x * BPT;
  uint64_t sum = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) sum += hv(b0 + q);
  uint64_t tot;
  const uint64_t excl = blk_excl_scan_u64(sum, s, &tot);
  total = tot;
  const double target = MASS ? tgt * (double)tot : tgt;
  int mine = 0x7fffffff;
  if ((double)excl < target && (double)(excl + sum) >= target) {  // at most one thread
    uint64_t cum = excl;
    int b = b0;
    while (b < b0 + BPT - 1 && (double)(cum + hv(b)) < target) cum += hv(b++);
    mine = b;
    s.bc_q[1] = cum;
  }
  bb = blk_min_i(mine, s);
  before = s.bc_q[1];
  __syncthreads();
  return bb != 0x7fffffff;
}

// Pass two: the order keys of the finite values z >= lo of distance bucket bb, staged in LDS (the list
// area).  Returns their number, or -1 when they do not fit.
template <class DT, bool SEG>
__device__ __forceinline__ int gp_gather(const SArgs& a, const SRow& R, SSm& s, float lo, float m, int bb) {
  uint32_t* keys = reinterpret_cast<uint32_t*>(r_gstage);
  if (threadIdx.x == 0) s.bc_i[2] = 0;
  __syncthreads();
  RowSrc<DT, SEG>{a, R, s}([&](float z) __attribute__((always_inline)) {
    if (z > -INFINITY && z >= lo && gp_dbucket(z, m) == bb) {
      const int i = atomicAdd(&s.bc_i[2], 1);
      if (i < GKCAP) keys[i] = f2key(z);
    }
  });
  __syncthreads();
  const int n = s.bc_i[2];
  __syncthreads();
  return n <= GKCAP ? n : -1;
}

// General path: the order key of the K-th largest finite value (counting duplicates), or 0 when there
// are fewer than K: a count over the distance buckets, then the exact selection among the values of
// the bucket holding it (over the whole row only when that bucket does not fit in LDS).
template <class DT, bool SEG>
__device__ __forceinline__ uint32_t gp_kth(const SArgs& a, const SRow& R, SSm& s, float m, int K) {
  int bb;
  uint64_t before, total;
  if (!gp_level1<false, DT, SEG>(a, R, s, -INFINITY, m, (double)K, bb, before, total)) return 0u;
  const int n = gp_gather<DT, SEG>(a, R, s, -INFINITY, m, bb);
  uint32_t* hist = reinterpret_cast<uint32_t*>(r_gstage) + GKCAP;
  if (n >= 0)
    return gp_kth_key(StagedSrc{reinterpret_cast<const uint32_t*>(r_gstage), n}, s, hist, K - (int)before);
  return gp_kth_key(RowSrc<DT, SEG>{a, R, s}, s, reinterpret_cast<uint32_t*>(s.c.gen), K);
}

// General path: the order key of the nucleus' closing group among the values z >= tau2 (the first
// group, in descending order, at which the cumulative mass reaches p times the mass of all of them),
// or 0 when the cumulative never reaches it: a mass over the distance buckets, then the exact
// selection inside the bucket where the cumulative crosses.
template <class DT, bool SEG>
__device__ __forceinline__ uint32_t gp_topp(const SArgs& a, const SRow& R, SSm& s, float tau2, float m, double p) {
  int bb;
  uint64_t before, total;
  if (!gp_level1<true, DT, SEG>(a, R, s, tau2, m, p, bb, before, total)) return 0u;
  const double target = p * (double)total;
  const int n = gp_gather<DT, SEG>(a, R, s, tau2, m, bb);
  if (n >= 0)
    return gp_topp_key(StagedSrc{reinterpret_cast<const uint32_t*>(r_gstage), n}, s, s.c.gen, tau2, m, target,
                       (double)before);
  return gp_topp_key(RowSrc<DT, SEG>{a, R, s}, s, s.c.gen, tau2, m, target, 0.0);
}

// The nucleus cut among the values z >= tau2 (as gp_topp), with the draw's per-chunk kept masses taken
// in the same passes: a value in a distance bucket above the crossing one is kept whatever the cut
// inside that bucket, so its mass goes to its chunk during the gather; the crossing bucket's values are
// staged with their positions and, once the cut is known, the kept ones join their chunks.  The sums are
// integers, so the masses equal those of a separate pass.  Returns false (nothing decided) when the
// cumulative never reaches the target or the bucket does not fit in LDS; the caller then selects and
// draws the separate way.
// Sub-bucket (0 .. GDB - 1) of a value inside distance bucket bb: the fraction of the bucket, GDB steps.
// fl(m - z) GD_SCALE is monotone in z and its distance from the integer bb is exact, so the sub-buckets
// order the bucket's values as the buckets order the row's.
__device__ __forceinline__ int gp_dsub(float z, float m, int bb) {
  const float d = __fmul_rn(__fsub_rn(m, z), GD_SCALE);
  const int sb = (int)__fmul_rn(__fsub_rn(d, (float)bb), (float)GDB);
  return sb < 0 ? 0 : (sb > GDB - 1 ? GDB - 1 : sb);
}

template <class DT, bool SEG>
__device__ __forceinline__ bool gp_topp_fused(const SArgs& a, const SRow& R, SSm& s, float tau2, float m, double p,
                                              float& tau, int& last) {
  int bb;
  uint64_t before, total;
  if (!gp_level1<true, DT, SEG>(a, R, s, tau2, m, p, bb, before, total)) return false;
  const double target = p * (double)total;
  uint64_t* ent = r_gstage;
  uint64_t* cm = s.cm;
  // refine: values of bucket bb with sub-bucket < sbb count as above the crossing, those of sub-bucket
  // sbb are staged (sbb = GDB: the whole bucket is staged)
  int sbb = GDB;
  for (int round = 0; round < 2; ++round) {
    for (int c = threadIdx.x; c < R.P; c += CT) cm[c] = 0;
    if (threadIdx.x == 0) s.bc_i[2] = 0;
    __syncthreads();
    int lastp = -1;
    for (int c = 0; c < R.P; ++c) {
      uint64_t acc = 0;
      for_chunk<DT, SEG>(a, R, s, c, [&](float z, int pos) __attribute__((always_inline)) {
        if (z > -INFINITY && z >= tau2) {
          const int b = gp_dbucket(z, m);
          const int sub = (b == bb && sbb < GDB) ? gp_dsub(z, m, bb) : GDB;
          if (b < bb || (b == bb && sub < sbb)) {
            const uint64_t w = mass_of(z, m);
            acc += w;
            if (w > 0) lastp = max(lastp, pos);
          } else if (b == bb && sub == sbb) {
            const int i = atomicAdd(&s.bc_i[2], 1);
            if (i < GKCAP2) ent[i] = ((uint64_t)f2key(z) << 32) | (uint32_t)pos;
          }
        }
      });
      if (acc) atomicAdd(reinterpret_cast<unsigned long long*>(&cm[c]), (unsigned long long)acc);
    }
    __syncthreads();
    const int n = s.bc_i[2];
    __syncthreads();
    if (n <= GKCAP2) {
      const uint32_t kk = gp_topp_key(StagedPairs{ent, n}, s, s.c.gen, tau2, m, target, (double)before);
      if (!kk) return false;  // not reached inside the staged values: cannot happen, decided the separate way
      tau = fmaxf(tau2, key2f(kk));
      for (int i = threadIdx.x; i < n; i += CT) {
        const uint64_t e = ent[i];
        const float z = key2f((uint32_t)(e >> 32));
        if (z >= tau) {
          const int pos = (int)(uint32_t)e;
          const uint64_t w = mass_of(z, m);
          atomicAdd(reinterpret_cast<unsigned long long*>(&cm[chunk_of(a, R, DT::VEC, pos)]), (unsigned long long)w);
          if (w > 0) lastp = max(lastp, pos);
        }
      }
      last = blk_max_i(lastp, s);  // its barriers also publish cm
      return true;
    }
    if (round == 1) return false;
    // the bucket does not fit: one pass for the mass histogram of its sub-buckets, then the crossing
    // sub-bucket becomes the staged part
    uint64_t* h64 = s.c.gen;
    for (int i = threadIdx.x; i < GDB; i += CT) h64[i] = 0;
    __syncthreads();
    RowSrc<DT, SEG>{a, R, s}([&](float z) __attribute__((always_inline)) {
      if (z > -INFINITY && z >= tau2 && gp_dbucket(z, m) == bb) {
        const uint64_t w = mass_of(z, m);
        if (w) atomicAdd(reinterpret_cast<unsigned long long*>(&h64[gp_dsub(z, m, bb)]), (unsigned long long)w);
      }
    });
    __syncthreads();
    constexpr int BPT = GDB / CT;
    const int i0 = (int)threadIdx.x * BPT;
    uint64_t sum = 0;
#pragma unroll
    for (int q = 0; q < BPT; ++q) sum += h64[i0 + q];
    uint64_t tot;
    const uint64_t excl = blk_excl_scan_u64(sum, s, &tot);
    int mine = 0x7fffffff;
    if ((double)before + (double)excl < target && (double)before + (double)(excl + sum) >= target) {
      uint64_t cum = excl;
      int i = i0;
      while (i < i0 + BPT - 1 && (double)before + (double)(cum + h64[i]) < target) cum += h64[i++];
      mine = i;
      s.bc_q[1] = cum;
    }
    const int sb = blk_min_i(mine, s);
    if (sb == 0x7fffffff) return false;
    before += s.bc_q[1];
    sbb = sb;
    __syncthreads();
  }
  return false;
}

// General path: kept set S = {finite z >= tau}; draws the token with target u * Z_S in ascending id.
// Returns the id (z in *zid).  masses_known: the per-chunk kept masses are already in s.cm and `last`
// is the last position of positive kept mass (the nucleus selection took them in its own pass).
template <class DT, bool SEG>
__device__ __forceinline__ int gp_draw(const SArgs& a, const SRow& R, SSm& s, float tau, float m, float u, float* zid,
                                       bool masses_known, int last) {
  constexpr int VEC = DT::VEC;
  const int P = R.P, t = threadIdx.x;
  uint64_t* cm = s.cm;  // per chunk mass
  if (!masses_known) {
    for (int c = t; c < P; c += CT) cm[c] = 0;
    __syncthreads();
    last = -1;
    for (int c = 0; c < P; ++c) {
      uint64_t acc = 0;
      for_chunk<DT, SEG>(a, R, s, c, [&](float z, int pos) __attribute__((always_inline)) {
        if (z > -INFINITY && z >= tau) {
          const uint64_t w = mass_of(z, m);
          acc += w;
          if (w > 0) last = max(last, pos);
        }
      });
      if (acc) atomicAdd(reinterpret_cast<unsigned long long*>(&cm[c]), (unsigned long long)acc);
    }
    last = blk_max_i(last, s);
  }
  uint64_t zs = 0;
  for (int c = 0; c < P; ++c) zs += cm[c];
  const double target = (double)u * (double)zs;
  // the chunk holding the first prefix above the target
  int cs = -1;
  uint64_t before = 0;
  for (int c = 0; c < P; ++c) {
    if ((double)(before + cm[c]) > target) { cs = c; break; }
    before += cm[c];
  }
  __syncthreads();
  int id = -1;
  float zf = -INFINITY;
  if (cs >= 0) {
    // chunk cs in ascending position, in batches of CT * GJ consecutive slots: thread t of a batch takes
    // GJ consecutive slots (thread 0 of the first batch also the unaligned head before them, the last
    // thread of the last batch the tail after them); each thread's kept mass, an exclusive scan in
    // thread order; the batch holding the crossing has its crossing thread walk its positions
    int64_t s0, s1;
    chunk_range(a, R, cs, s0, s1);
    const int ns = (int)(s1 - s0);
    const int64_t e_base = (int64_t)R.head + (s0 - 1) * VEC;
    float hx[8];
    int hn = 0, hp0 = 0;
    if (t == 0 && cs == 0) { hn = R.head; hp0 = 0; }
    if (t == CT - 1 && cs == P - 1) { hn = R.V - R.tail_lo; hp0 = R.tail_lo; }
#pragma unroll
    for (int q = 0; q < 8; ++q) hx[q] = hn > 0 ? load_elem<DT, SEG>(a, R, hp0 + min(q, hn - 1)) : 0.0f;
    if (R.pen_on) {
      uint32_t fl = 0;
      const int32_t none[1] = {0};
      build_overlay<0>(a, R, s, cs, s0, s1, VEC, none, &fl);
    }
    const float r = R.r;
    auto value = [&](float x, int pos) __attribute__((always_inline)) -> float {
      if (R.pen_on) {
        const int rk = overlay_rank(s, (int)(pos - e_base));
        if (rk >= 0) x = penalise_cv(x, s.c.p.xval[rk], R.rep, R.freq, R.pres);
      }
      return canon(x, r);
    };
    auto kept = [&](float z) __attribute__((always_inline)) -> uint64_t {
      return (z > -INFINITY && z >= tau) ? mass_of(z, m) : 0ull;
    };
    const int nbat = max(1, (ns + CT * GJ - 1) / (CT * GJ));  // a chunk of head and tail alone: one batch
    uint64_t cum0 = before;
    for (int bt = 0; bt < nbat; ++bt) {
      const int b0 = bt * CT * GJ;
      const int nb = min(ns - b0, CT * GJ);
      uint4 d[GJ];
      static_for<GJ>([&](auto J) {  // unconditional loads (clamped into the batch, or the records' first word)
        constexpr int j = decltype(J)::value;
        d[j] = *(nb > 0 ? slot_ptr<DT, SEG>(a, R, s0 + b0 + min(t * GJ + j, nb - 1))
                        : reinterpret_cast<const uint4*>(a.rec));
      });
      const bool head_here = t == 0 && cs == 0 && bt == 0;
      const bool tail_here = t == CT - 1 && cs == P - 1 && bt == nbat - 1;
      // walk(f): this thread's positions of the batch in ascending order
      auto walk = [&](auto&& f) __attribute__((always_inline)) {
        if (head_here)
          for (int q = 0; q < hn; ++q) f(value(hx[q], hp0 + q), hp0 + q);
        static_for<GJ>([&](auto J) {
          constexpr int j = decltype(J)::value;
          if (t * GJ + j < nb) {
            const int p0 = R.head + (int)(s0 + b0 + t * GJ + j) * VEC;
#pragma unroll
            for (int e = 0; e < VEC; ++e) f(value(elem<DT>(d[j], e), p0 + e), p0 + e);
          }
        });
        if (tail_here)
          for (int q = 0; q < hn; ++q) f(value(hx[q], hp0 + q), hp0 + q);
      };
      uint64_t mine = 0;
      walk([&](float z, int) __attribute__((always_inline)) { mine += kept(z); });
      uint64_t tot;
      uint64_t cum = cum0 + blk_excl_scan_u64(mine, s, &tot);
      int found = 0x7fffffff;
      float zfound = -INFINITY;
      if ((double)cum <= target && (double)(cum + mine) > target) {
        bool done = false;
        walk([&](float z, int pos) __attribute__((always_inline)) {
          if (!done) {
            cum += kept(z);
            if ((double)cum > target) {
              done = true;
              found = pos;
              zfound = z;
            }
          }
        });
      }
      const int idb = blk_min_i(found, s);
      if (found == idb && idb != 0x7fffffff) s.bc_f[0] = zfound;
      __syncthreads();
      if (idb != 0x7fffffff) {  // the same for every thread
        id = idb;
        zf = s.bc_f[0];
        break;
      }
      cum0 += tot;
    }
    __syncthreads();  // the overlay and bc_f are free again
  }
  if (id < 0) {
    id = last;
    // its value: a re-read of its chunk
    if (threadIdx.x == 0) s.bc_f[0] = -INFINITY;
    __syncthreads();
    if (id >= 0) {
      for_chunk<DT, SEG>(a, R, s, chunk_of(a, R, VEC, id), [&](float z, int pos) __attribute__((always_inline)) {
        if (pos == id && z > -INFINITY) s.bc_f[0] = z;  // a penalised id is also visited as -inf
      });
    }
    __syncthreads();
    zf = s.bc_f[0];
    __syncthreads();
  }
  *zid = zf;
  return id;
}

// The general path rebuilds a chunk's penalty overlay for every re-read: the row's output history,
// copied to LDS when the kernel starts, is grouped by the chunk its ids fall in, so that a rebuild
// reads only its chunk's ids.  Every thread of the workgroup calls it.
template <class DT>
__device__ __forceinline__ void stage_history(const SArgs& a, const SRow& R, SSm& s) {
  const int t = threadIdx.x;
  const int64_t nh = R.h_hi - R.h_lo;
  if (s.hst_on) {
    // the ids grouped by the chunk they fall in (a counting sort; the order inside a group does not
    // matter, its ids are counted by atomics); ids outside [0, V) are left out (the chunk kernel has
    // flagged them already)
    constexpr int Q = HSTAGE / CT;
    int32_t v[Q];
    static_for<Q>([&](auto I) {
      constexpr int q = decltype(I)::value;
      v[q] = r_hstage[min(t + q * CT, (int)nh - 1)];
    });
    if (t <= R.P) s.hoff[t] = 0;
    __syncthreads();
    int cq[Q];
    static_for<Q>([&](auto I) {
      constexpr int q = decltype(I)::value;
      const int id = v[q];
      cq[q] = (t + q * CT < nh && id >= 0 && id < R.V) ? chunk_of(a, R, DT::VEC, id) : -1;
      if (cq[q] >= 0) atomicAdd(&s.hoff[cq[q] + 1], 1);
    });
    __syncthreads();
    if (t == 0) {
      for (int c = 0; c < R.P; ++c) {
        s.hcur[c] = s.hoff[c];
        s.hoff[c + 1] += s.hoff[c];
      }
    }
    __syncthreads();
    static_for<Q>([&](auto I) {
      constexpr int q = decltype(I)::value;
      if (cq[q] >= 0) r_hstage[atomicAdd(&s.hcur[cq[q]], 1)] = v[q];
    });
  }
  __syncthreads();
}

// The general path of a row with no small kept-set bound: the top-k threshold, the nucleus and the draw
// over re-reads of the row.  Returns (id, bits of its z).
template <class DT, bool SEG>
__device__ __forceinline__ int2 resolve_general(const SArgs& a, const SRow& R, SSm& s, float m, float tau_m, float u) {
  stage_history<DT>(a, R, s);
  float tau_k = -INFINITY;
  if (R.kon) {
    const uint32_t kk = gp_kth<DT, SEG>(a, R, s, m, R.k);
    tau_k = kk ? key2f(kk) : -INFINITY;
  }
  const float tau2 = fmaxf(tau_k, tau_m);
  float tau = tau2;
  bool fused = false;
  int last = -1;
  if (R.topp_on) {
    if (!(R.p > 0.0f)) {
      tau = m;  // p <= 0: the top group only
    } else {
      fused = gp_topp_fused<DT, SEG>(a, R, s, tau2, m, (double)R.p, tau, last);
      if (!fused) {
        const uint32_t kk = gp_topp<DT, SEG>(a, R, s, tau2, m, (double)R.p);
        tau = kk ? fmaxf(tau2, key2f(kk)) : tau2;
      }
    }
  }
  float zid = -INFINITY;
  const int id = gp_draw<DT, SEG>(a, R, s, tau, m, u, &zid, fused, last);
  return make_int2(id, __float_as_int(zid));
}

// ----------------------------------------------------------------------------------------------
// The row's resolution by its last chunk workgroup
// ----------------------------------------------------------------------------------------------
template <class DT, bool SEG>
__device__ __forceinline__ void resolve_row(const SArgs& a, const SRow& R, SSm& s) {
  const int t = threadIdx.x, P = R.P;
  const int64_t row = R.row;
  const int nt = a.n_top;
  // ---- one round trip: the chunk records, the row's uniform and the heads of the chunk lists ----
  Spec sp;
  sp.E = nt;
  if (R.kon) sp.E = max(sp.E, min(R.k + 1, LCAPC));  // the k-th entry too, for the tie test
  sp.on = sp.E > 0 && P * sp.E <= SPQ * CT;
  if (sp.on) {
    const uint64_t* base = a.lists + (row * P) * (int64_t)LCAPC;
#pragma unroll
    for (int q = 0; q < SPQ; ++q) {
      const int f = t + q * CT;
      sp.v[q] = 0;
      if (f < P * sp.E) {
        const int c = f / sp.E;
        sp.v[q] = base[(int64_t)c * LCAPC + (f - c * sp.E)];
      }
    }
  }
  if (t < P) s.pub[t] = rec_load(a.rec + (row * P + t) * REC_WORDS);
  float u = 0.0f;
  if (a.rng_on) {
    const uint64_t seq = a.seq_ids ? (uint64_t)a.seq_ids[row] : (uint64_t)row;
    u = philox_uniform(a.rng_seed, a.rng_step, seq);
  } else {
    u = a.uniforms[row];
  }
  __syncthreads();
  // row totals, in chunk order (every thread computes the same)
  float m = -INFINITY, mref = MREF0, S = 0.0f;
  uint32_t flags = R.flags;
  bool fin = false, over_any = false;
  int argpos = -1;
  for (int c = 0; c < P; ++c) {
    const ChunkPub& q = s.pub[c];
    m = fmaxf(m, q.zmax);
    lse_add(mref, S, q.mref, q.s);
    flags |= q.flags & (FLAG_BAD_INPUT | FLAG_LIMIT);
    fin = fin || (q.flags & PUB_FINITE);
    over_any = over_any || (q.flags & PUB_OVER);
  }
  for (int c = 0; c < P; ++c)
    if (s.pub[c].zmax == m) { argpos = s.pub[c].argpos; break; }
  if (a.st_flags) flags |= a.st_flags[row] & (FLAG_BAD_INPUT | FLAG_BAD_PARAM | FLAG_LIMIT);
  const bool empty = !fin;
  if (empty) flags |= FLAG_EMPTY;
  const double L = log((double)S) - ((double)m * (double)L2E - (double)mref) * LN2;

  // ---- top-n: the n largest keys of the lists (each list holds its chunk's top n), by counted rank ----
  if (nt > 0) {
    if (t < nt) {
      s.top_id[t] = -1;
      s.top_lp[t] = -INFINITY;
    }
    if (!empty) {
      float lo = INFINITY;
      for (int c = 0; c < P; ++c) lo = fminf(lo, s.pub[c].qn);
      const int ns = stage_entries(a, R, s, sp, lo, nt, MSTAGE, false);
      for (int f = t; f < ns; f += CT) {
        const uint64_t key = s.key[f];
        const int rk = count_above(s.key, ns, key);
        if (rk < nt) {
          s.top_id[rk] = cand_pos(key);
          s.top_lp[rk] = (float)((double)cand_z(key) - (double)m - L);
        }
      }
    }
    __syncthreads();
    if (t < nt) {
      a.out_top_ids[row * nt + t] = s.top_id[t];
      a.out_top_logprobs[row * nt + t] = s.top_lp[t];
    }
  }

  int id = -1;
  float zid = -INFINITY;
  bool defer = false;
  uint64_t defer_w[4] = {0, 0, 0, 0};
  if (empty) {
    id = -1;
  } else if (R.greedy) {
    id = argpos;
    zid = m;
  } else {
    // ---- the kept set from the lists when it is small; otherwise the general path ----
    const bool s2b = R.kon || R.minp_on;
    const float tau_m = R.minp_on ? __fadd_rn(m, (float)log((double)R.minp)) : -INFINITY;
    bool general = !s2b || over_any;
    // kept set S2: A[i] = (order key of z << 32) | mass, Bk[i] = (position << 32) | mass kept by the
    // nucleus; masses 2^((z - m) L2E) in units of 2^-31
    uint64_t* A = s.key + (MSTAGE - 2 * MCAP);
    uint64_t* Bk = s.key + (MSTAGE - MCAP);
    int n2 = 0;
    if (!general) {
      float tau2 = tau_m;
      const int imax = R.kon ? min(R.k, LCAPC) : LCAPC;
      float zthr = tau_m;
      if (R.kon) {
        float lo = INFINITY;
        for (int c = 0; c < P; ++c) lo = fminf(lo, s.pub[c].qk);
        zthr = fmaxf(zthr, lo);
      }
      int ns = stage_entries(a, R, s, sp, zthr, imax, MSTAGE - 2 * MCAP, true);
      if (ns < 0) {
        general = true;
      } else {
        if (R.kon) {
          if (t == 0) s.bc_f[1] = -INFINITY;
          __syncthreads();
          for (int f = t; f < ns; f += CT)
            if (count_above(s.key, ns, s.key[f]) == R.k - 1) s.bc_f[1] = cand_z(s.key[f]);
          __syncthreads();
          tau2 = fmaxf(tau2, s.bc_f[1]);
        }
        // a list cut off at imax whose first entry left out would be kept (a tie at tau_k): the kept
        // set is then every list entry z >= tau2 -- no list is over capacity here, and each holds all
        // of its chunk's values above the chunk's bound, which is at most the chunk's K-th largest
        // and so at most tau2
        bool cutkept = false;
        for (int c = 0; c < P; ++c)
          if (s.cut[c] && __int_as_float(s.cnt[c]) >= tau2) cutkept = true;
        if (cutkept) {
          ns = stage_entries(a, R, s, sp, tau2, LCAPC, MSTAGE - 2 * MCAP, false);
          cutkept = ns < 0;
          if (ns < 0) ns = 0;
        }
        if (t == 0) s.bc_i[2] = 0;
        __syncthreads();
        for (int f = t; f < ns; f += CT) {
          const uint64_t key = s.key[f];
          const float z = cand_z(key);
          if (z >= tau2) {
            const int idx = atomicAdd(&s.bc_i[2], 1);
            if (idx < MCAP) {
              const uint32_t w = (uint32_t)(__builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(z, m), L2E)) * 2147483648.0f);
              A[idx] = ((uint64_t)f2key(z) << 32) | w;
              Bk[idx] = ((uint64_t)(uint32_t)cand_pos(key) << 32) | w;
            }
          }
        }
        __syncthreads();
        n2 = s.bc_i[2];
        if (n2 > MCAP || n2 == 0 || cutkept) general = true;
      }
    }
    if (!general) {
      // nucleus: keep every entry whose strictly larger values carry less than p of the S2 mass
      uint64_t z2 = 0;
      for (int i = t; i < n2; i += CT) z2 += (uint32_t)A[i];
      z2 = blk_sum_u64(z2, s);
      const double T = (double)R.p * (double)z2;
      uint64_t zsum = 0;
      for (int i = t; i < n2; i += CT) {
        const uint64_t ai = A[i];
        bool keep = true;
        if (R.topp_on) {
          const uint32_t zk = (uint32_t)(ai >> 32);
          uint64_t above = 0;
#pragma unroll 8
          for (int j = 0; j < n2; ++j) {
            const uint64_t aj = A[j];
            above += ((uint32_t)(aj >> 32) > zk) ? (uint32_t)aj : 0u;
          }
          keep = above == 0 || (double)above < T;
        }
        if (!keep) Bk[i] &= 0xffffffff00000000ull;
        zsum += keep ? (uint32_t)ai : 0u;
      }
      zsum = blk_sum_u64(zsum, s);
      // inverse CDF in ascending token id: the first kept position whose prefix mass exceeds u Z_S
      const double target = (double)u * (double)zsum;
      int found = 0x7fffffff, lastp = -1;
      for (int i = t; i < n2; i += CT) {
        const uint64_t bi = Bk[i];
        if ((uint32_t)bi == 0) continue;
        const uint32_t pi = (uint32_t)(bi >> 32);
        lastp = max(lastp, (int)pi);
        uint64_t pre = 0;
#pragma unroll 8
        for (int j = 0; j < n2; ++j) {
          const uint64_t bj = Bk[j];
          pre += ((uint32_t)(bj >> 32) <= pi) ? (uint32_t)bj : 0u;
        }
        if ((double)pre > target) found = min(found, (int)pi);
      }
      found = blk_min_i(found, s);
      lastp = blk_max_i(lastp, s);
      id = found != 0x7fffffff ? found : lastp;
      if (t == 0) s.bc_f[2] = -INFINITY;
      __syncthreads();
      for (int i = t; i < n2; i += CT)
        if ((int)(uint32_t)(Bk[i] >> 32) == id) s.bc_f[2] = key2f((uint32_t)(A[i] >> 32));
      __syncthreads();
      zid = s.bc_f[2];
    } else if (!R.kon) {
      // no top-k threshold to select: the chunk-parallel launches take the row from here
      defer = true;
      if (t == 0) {
        const bool topp = R.topp_on && R.p > 0.0f;
        const float lo = (R.topp_on && !(R.p > 0.0f)) ? m : tau_m;  // p <= 0: the top group only
        defer_w[0] = RS_DEFER | (topp ? RS_TOPP : 0);
        defer_w[1] = (uint64_t)__float_as_uint(m) | ((uint64_t)__float_as_uint(lo) << 32);
        defer_w[2] = (uint64_t)__float_as_uint(u) | ((uint64_t)__float_as_uint(R.p) << 32);
        defer_w[3] = (uint64_t)__double_as_longlong(L);
      }
    } else {
      const int2 r2 = resolve_general<DT, SEG>(a, R, s, m, tau_m, u);
      id = r2.x;
      zid = __int_as_float(r2.y);
    }
  }
  // leave the workspace as it was found: zero the row's chunk records and lists
  {
    uint64_t* lbase = a.lists + (row * P) * (int64_t)LCAPC;
    for (int c = 0; c < P; ++c) {
      const int n = min(s.pub[c].n_list, LCAPC);
      for (int i = t; i < n; i += CT) lbase[(int64_t)c * LCAPC + i] = 0;
    }
    uint64_t* rw = a.rec + row * P * REC_WORDS;
    for (int i = t; i < P * REC_WORDS; i += CT) rw[i] = 0;
  }
  if (t == 0) {
    if (a.out_flags) a.out_flags[row] = flags;
    if (defer) {
      uint64_t* rs = a.rstate + row * RS_WORDS;
      for (int i = 0; i < 4; ++i) rs[i] = defer_w[i];
      a.dq[2 + atomicAdd(&a.dq[0], 1)] = (int32_t)row;
    } else {
      float lp = -INFINITY;
      if (!empty) lp = (float)((double)zid - (double)m - L);
      a.out_ids[row] = id;
      a.out_logprobs[row] = lp;
      if (a.next_tokens) {
        const int32_t dst = a.backfill_dest[row];
        if (dst >= 0 && (int64_t)dst < a.next_len) a.next_tokens[dst] = id;
      }
    }
  }
}

// ----------------------------------------------------------------------------------------------
// Deferred rows: the general path of a row with no top-k, spread over its chunks.  The resolution
// kernel leaves such a row's maximum m, the lower cut lo (min-p, or m for p <= 0), its uniform, p and
// log-normaliser in the row's state.  Then
//   k_gen_a (per chunk): the chunk's kept mass (values >= lo, fixed-point masses against
//     m) and, for a nucleus, its mass per distance bucket, into the chunk's list slot;
//   k_gen_b (per chunk, nucleus rows): every chunk of the row merges the histograms to the
//     bucket where the cumulative reaches p times the total; the chunk sums its mass above that bucket
//     and stages the bucket's values (up to SCAP) and the bucket's mass per sub-bucket;
//   k_gen_s (per chunk, rows where a chunk had more than SCAP of the bucket's values):
//     every chunk merges the sub-bucket masses to the crossing sub-bucket and stages its values instead;
//   k_gen_c (per row): the cut inside the staged bucket or sub-bucket, the per-chunk kept
//     masses and the draw over the crossing chunk; it writes the row's id and logprob and zeroes what
//     the row used.
// The resolution kernel appends each deferred row to a list in the workspace; these launches walk that
// list, one workgroup per (row, chunk) or per row at a time, so a call without deferred rows costs four
// small grids that find the list empty.
// Every sum is an integer sum of the same masses the single-workgroup general path takes and the staged
// sets are the same, so the result is the same; a row whose staging does not fit takes that path (or a
// pass over the row for its crossing sub-bucket) in k_gen_c.
// ----------------------------------------------------------------------------------------------
struct Deferred {
  bool on, topp;
  float m, lo, u, p;
  double L;
};
__device__ __forceinline__ Deferred deferred_of(const SArgs& a, int64_t row) {
  const uint64_t* rs = a.rstate + row * RS_WORDS;
  Deferred d;
  const uint64_t w0 = rs[0];
  d.on = (w0 & RS_DEFER) != 0;
  d.topp = (w0 & RS_TOPP) != 0;
  d.m = d.lo = d.u = d.p = 0.0f;
  d.L = 0.0;
  if (d.on) {
    const uint64_t w1 = rs[1], w2 = rs[2];
    d.m = __uint_as_float((uint32_t)w1);
    d.lo = __uint_as_float((uint32_t)(w1 >> 32));
    d.u = __uint_as_float((uint32_t)w2);
    d.p = __uint_as_float((uint32_t)(w2 >> 32));
    d.L = __longlong_as_double((long long)rs[3]);
  }
  return d;
}

// The row's distance-bucket masses summed over its chunks' histograms (in their list slots), and the
// bucket where the cumulative, from the top, reaches p times the total (as the single-workgroup first
// level finds it).  Returns false when it is never reached.
__device__ __forceinline__ bool merge_hists(const SArgs& a, const SRow& R, SSm& s, double p, int& bb,
                                            uint64_t& before, uint64_t& total) {
  constexpr int BPT = GDB / CT;
  const uint64_t* base = a.lists + (R.row * R.P) * (int64_t)LCAPC;
  const int b0 = (int)threadIdx.x * BPT;
  uint64_t hv[BPT];
  uint64_t sum = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    uint64_t v = 0;
    for (int c = 0; c < R.P; ++c) v += base[(int64_t)c * LCAPC + b0 + q];
    hv[q] = v;
    sum += v;
  }
  uint64_t tot;
  const uint64_t excl = blk_excl_scan_u64(sum, s, &tot);
  total = tot;
  const double target = p * (double)tot;
  int mine = 0x7fffffff;
  if ((double)excl < target && (double)(excl + sum) >= target) {  // at most one thread
    uint64_t cum = excl;
    int q = 0;
    while (q < BPT - 1 && (double)(cum + hv[q]) < target) cum += hv[q++];
    mine = b0 + q;
    s.bc_q[1] = cum;
  }
  bb = blk_min_i(mine, s);
  before = s.bc_q[1];
  __syncthreads();
  return bb != 0x7fffffff;
}

// The crossing bucket's sub-bucket where the cumulative, continued from `before`, reaches p times the
// total (as the single-workgroup second round finds it), from the chunks' sub-bucket masses; the mass of
// the sub-buckets above it in *cum.  Returns 0x7fffffff when it is never reached.
__device__ __forceinline__ int merge_subs(const SArgs& a, const SRow& R, SSm& s, double target,
                                          uint64_t before, uint64_t* cum_out) {
  constexpr int BPT = GDB / CT;
  const int i0 = (int)threadIdx.x * BPT;
  uint64_t hv[BPT];
  uint64_t sum = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    uint64_t v = 0;
    for (int c = 0; c < R.P; ++c) v += a.stg[(R.row * R.P + c) * (int64_t)SSTRIDE + SCAP + i0 + q];
    hv[q] = v;
    sum += v;
  }
  uint64_t tot;
  const uint64_t excl = blk_excl_scan_u64(sum, s, &tot);
  int mine = 0x7fffffff;
  if ((double)before + (double)excl < target && (double)before + (double)(excl + sum) >= target) {
    uint64_t cum = excl;
    int q = 0;
    while (q < BPT - 1 && (double)before + (double)(cum + hv[q]) < target) cum += hv[q++];
    mine = i0 + q;
    s.bc_q[1] = cum;
  }
  const int sbb = blk_min_i(mine, s);
  *cum_out = s.bc_q[1];
  __syncthreads();
  return sbb;
}

// Whether every chunk of the row published its crossing-bucket staging (k_gen_b), and whether each
// holds its whole share (at most SCAP values) with at most GKCAP2 in all.  Uniform over the workgroup.
struct StageCounts {
  bool all_written, all_fit;
  int total;
};
__device__ __forceinline__ StageCounts stage_counts(const SArgs& a, const SRow& R) {
  StageCounts r{true, true, 0};
  const uint64_t* rec = a.rec + (R.row * R.P) * (int64_t)REC_WORDS;
  for (int c = 0; c < R.P; ++c) {
    const uint64_t w2 = rec[c * REC_WORDS + 2];
    if (!w2) {
      r.all_written = false;
      r.all_fit = false;
      continue;
    }
    const int nc = (int)(w2 - 1);
    if (nc > SCAP) r.all_fit = false;
    r.total += min(nc, SCAP);
  }
  return r;
}

template <class DT, bool SEG>
__device__ __forceinline__ void gen_a_item(const SArgs& a, SSm& s, int64_t row, int c) {
  const int t = threadIdx.x;
  const int64_t L = row * a.P + c;
  const Deferred d = deferred_of(a, row);
  if (!d.on) return;
  SRow R;
  row_setup<DT, SEG>(a, row, c, R);
  int32_t hreg[16];
  history_regs<16>(a, R, hreg);
  if (t == 0) s.hst_on = 0;
  uint64_t* h64 = s.c.gen;
  for (int b = t; b < GDB; b += CT) h64[b] = 0;
  __syncthreads();
  uint64_t acc = 0;
  int last = -1;
  const float m = d.m, lo = d.lo;
  const bool topp = d.topp;
  for_chunk_h<DT, SEG, 16>(a, R, s, c, hreg, [&](float z, int pos) __attribute__((always_inline)) {
    if (z > -INFINITY && z >= lo) {
      const uint64_t w = mass_of(z, m);
      if (w) {
        acc += w;
        last = max(last, pos);
        if (topp) atomicAdd(reinterpret_cast<unsigned long long*>(&h64[gp_dbucket(z, m)]), (unsigned long long)w);
      }
    }
  });
  acc = blk_sum_u64(acc, s);
  last = blk_max_i(last, s);
  if (topp) {
    uint64_t* lst = a.lists + L * (int64_t)LCAPC;
    for (int b = t; b < GDB; b += CT) lst[b] = h64[b];
  }
  if (t == 0) {
    a.rec[L * REC_WORDS + 0] = acc;
    a.rec[L * REC_WORDS + 1] = (uint64_t)(uint32_t)last;
  }
}

template <class DT, bool SEG>
__device__ __forceinline__ void gen_b_item(const SArgs& a, SSm& s, int64_t row, int c) {
  const int t = threadIdx.x;
  const int64_t L = row * a.P + c;
  const Deferred d = deferred_of(a, row);
  if (!d.on || !d.topp) return;
  SRow R;
  row_setup<DT, SEG>(a, row, c, R);
  int32_t hreg[16];
  history_regs<16>(a, R, hreg);
  if (t == 0) {
    s.hst_on = 0;
    s.n_list = 0;
  }
  int bb;
  uint64_t before, total;
  if (!merge_hists(a, R, s, (double)d.p, bb, before, total)) return;  // the same in every chunk
  uint64_t acc = 0;
  int last = -1;
  const float m = d.m, lo = d.lo;
  uint64_t* stg = a.stg + L * (int64_t)SSTRIDE;
  uint64_t* sub = s.c.list;  // the crossing bucket's mass per sub-bucket
  for (int i = t; i < GDB; i += CT) sub[i] = 0;
  __syncthreads();
  for_chunk_h<DT, SEG, 16>(a, R, s, c, hreg, [&](float z, int pos) __attribute__((always_inline)) {
    if (z > -INFINITY && z >= lo) {
      const int b = gp_dbucket(z, m);
      if (b < bb) {
        const uint64_t w = mass_of(z, m);
        if (w) {
          acc += w;
          last = max(last, pos);
        }
      } else if (b == bb) {
        const int i = atomicAdd(&s.n_list, 1);
        if (i < SCAP) stg[i] = ((uint64_t)f2key(z) << 32) | (uint32_t)pos;
        const uint64_t w = mass_of(z, m);
        if (w) atomicAdd(reinterpret_cast<unsigned long long*>(&sub[gp_dsub(z, m, bb)]), (unsigned long long)w);
      }
    }
  });
  acc = blk_sum_u64(acc, s);
  last = blk_max_i(last, s);  // its barriers also publish n_list and sub
  for (int i = t; i < GDB; i += CT) stg[SCAP + i] = sub[i];
  if (t == 0) {
    a.rec[L * REC_WORDS + 2] = (uint64_t)(uint32_t)s.n_list + 1;  // + 1: written
    a.rec[L * REC_WORDS + 3] = acc;
    a.rec[L * REC_WORDS + 4] = (uint64_t)(uint32_t)last;
  }
}

// Rows whose crossing bucket put more than SCAP values into some chunk: every chunk merges the chunks'
// sub-bucket masses to the crossing sub-bucket and stages that sub-bucket's values in place of the
// bucket's (records words 5 and 6: their count + 1 and the last position kept with positive mass
// among the sub-buckets above it).
template <class DT, bool SEG>
__device__ __forceinline__ void gen_s_item(const SArgs& a, SSm& s, int64_t row, int c) {
  const int t = threadIdx.x;
  const int64_t L = row * a.P + c;
  const Deferred d = deferred_of(a, row);
  if (!d.on || !d.topp) return;
  SRow R;
  row_setup<DT, SEG>(a, row, c, R);
  const StageCounts sc = stage_counts(a, R);
  if (!sc.all_written || sc.all_fit) return;  // k_gen_c finishes these rows without it
  int32_t hreg[16];
  history_regs<16>(a, R, hreg);
  if (t == 0) {
    s.hst_on = 0;
    s.n_list = 0;
  }
  int bb;
  uint64_t before, total;
  if (!merge_hists(a, R, s, (double)d.p, bb, before, total)) return;
  uint64_t cum;
  const int sbb = merge_subs(a, R, s, (double)d.p * (double)total, before, &cum);
  if (sbb == 0x7fffffff) return;
  const float m = d.m, lo = d.lo;
  uint64_t* stg = a.stg + L * (int64_t)SSTRIDE;
  int lastp = -1;
  for_chunk_h<DT, SEG, 16>(a, R, s, c, hreg, [&](float z, int pos) __attribute__((always_inline)) {
    if (z > -INFINITY && z >= lo && gp_dbucket(z, m) == bb) {
      const int sb = gp_dsub(z, m, bb);
      if (sb < sbb) {
        if (mass_of(z, m) > 0) lastp = max(lastp, pos);
      } else if (sb == sbb) {
        const int i = atomicAdd(&s.n_list, 1);
        if (i < SCAP) stg[i] = ((uint64_t)f2key(z) << 32) | (uint32_t)pos;
      }
    }
  });
  lastp = blk_max_i(lastp, s);  // its barriers also publish n_list
  if (t == 0) {
    a.rec[L * REC_WORDS + 5] = (uint64_t)(uint32_t)s.n_list + 1;
    a.rec[L * REC_WORDS + 6] = (uint64_t)(uint32_t)lastp;
  }
}

template <class DT, bool SEG>
__device__ __forceinline__ void gen_c_item(const SArgs& a, SSm& s, int64_t row) {
  const int t = threadIdx.x;
  const Deferred d = deferred_of(a, row);
  if (!d.on) return;
  SRow R;
  row_setup<DT, SEG>(a, row, 0, R);
  const int P = R.P;
  if (t == 0) s.hst_on = 0;
  // before a pass over the whole row: the output history to LDS, grouped by chunk, for the overlay
  // rebuilds (the draw's walk over one chunk reads its ids from memory)
  auto history_to_lds = [&]() __attribute__((always_inline)) {
    const int64_t nh = R.h_hi - R.h_lo;
    if (R.pen_on && nh > 0 && nh <= HSTAGE) {
      constexpr int Q = HSTAGE / CT;
      int32_t v[Q];
      static_for<Q>([&](auto I) {  // every load in flight before any is stored
        constexpr int q = decltype(I)::value;
        v[q] = a.prm.hist_ids[R.h_lo + min((int64_t)(t + q * CT), nh - 1)];
      });
      static_for<Q>([&](auto I) {
        constexpr int q = decltype(I)::value;
        if (t + q * CT < nh) r_hstage[t + q * CT] = v[q];
      });
      if (t == 0) s.hst_on = 1;
    }
    __syncthreads();
    stage_history<DT>(a, R, s);
  };
  __syncthreads();
  const uint64_t* rec = a.rec + (row * P) * (int64_t)REC_WORDS;
  const float m = d.m, lo = d.lo;
  float tau = lo;
  int last = -1;
  bool fast = true;
  if (!d.topp) {
    if (t < P) {
      s.cm[t] = rec[t * REC_WORDS + 0];
      s.cnt[t] = (int32_t)(uint32_t)rec[t * REC_WORDS + 1];
    }
    __syncthreads();
    for (int c = 0; c < P; ++c) last = max(last, s.cnt[c]);
  } else {
    int bb;
    uint64_t before, total;
    fast = merge_hists(a, R, s, (double)d.p, bb, before, total);
    bool overfull = false;     // the crossing bucket's values did not fit the staging
    bool staged_all = false;   // but every chunk's share of them is staged
    int n = 0;
    if (fast) {
      if (t == 0) {
        int off = 0;
        bool ok = true;
        for (int c = 0; c < P; ++c) {
          const uint64_t w2 = rec[c * REC_WORDS + 2];
          const int nc = w2 ? (int)(w2 - 1) : -1;
          if (nc < 0 || nc > SCAP) ok = false;
          s.cut[c] = off;  // where chunk c's entries start
          s.cnt[c] = nc < 0 ? 0 : min(nc, SCAP);
          off += s.cnt[c];
        }
        s.bc_i[0] = ok && off <= GKCAP2 ? off : -1;
        s.bc_i[1] = ok ? 1 : 0;  // every chunk staged its whole crossing bucket
      }
      __syncthreads();
      n = s.bc_i[0];
      staged_all = s.bc_i[1] != 0;
      __syncthreads();
      fast = n >= 0;
      overfull = !fast;
    }
    if (fast) {
      uint64_t* ent = r_gstage;
      for (int c = 0; c < P; ++c) {
        const uint64_t* src = a.stg + (row * P + c) * (int64_t)SSTRIDE;
        for (int i = t; i < s.cnt[c]; i += CT) ent[s.cut[c] + i] = src[i];
      }
      __syncthreads();
      const uint32_t kk = gp_topp_key(StagedPairs{ent, n}, s, s.c.gen, lo, m, (double)d.p * (double)total,
                                      (double)before);
      fast = kk != 0;
      if (fast) {
        tau = fmaxf(lo, key2f(kk));
        if (t < P) s.cm[t] = rec[t * REC_WORDS + 3];
        int lastp = -1;
        for (int c = 0; c < P; ++c) lastp = max(lastp, (int)(uint32_t)rec[c * REC_WORDS + 4]);
        __syncthreads();
        for (int i = t; i < n; i += CT) {
          const uint64_t e = ent[i];
          const float z = key2f((uint32_t)(e >> 32));
          if (z >= tau) {
            const int pos = (int)(uint32_t)e;
            const uint64_t w = mass_of(z, m);
            atomicAdd(reinterpret_cast<unsigned long long*>(&s.cm[chunk_of(a, R, DT::VEC, pos)]), (unsigned long long)w);
            if (w > 0) lastp = max(lastp, pos);
          }
        }
        last = blk_max_i(lastp, s);  // its barriers also publish cm
      }
    }
    if (overfull) {
      // the crossing bucket did not fit the staging: its sub-buckets (GDB steps of the bucket, each
      // chunk's masses merged) give the sub-bucket where the cumulative crosses; one pass over the row
      // stages that sub-bucket's values (a comparison per value, masses only inside bucket bb)
      bool all = true;
      for (int c = 0; c < P; ++c) all = all && rec[c * REC_WORDS + 2] != 0;
      if (all) {
        constexpr int BPT = GDB / CT;
        const int i0 = t * BPT;
        uint64_t hv[BPT];
        uint64_t sum = 0;
#pragma unroll
        for (int q = 0; q < BPT; ++q) {
          uint64_t v = 0;
          for (int c = 0; c < P; ++c) v += a.stg[(row * P + c) * (int64_t)SSTRIDE + SCAP + i0 + q];
          hv[q] = v;
          sum += v;
        }
        uint64_t tot;
        const uint64_t excl = blk_excl_scan_u64(sum, s, &tot);
        const double target = (double)d.p * (double)total;
        int mine = 0x7fffffff;
        if ((double)before + (double)excl < target && (double)before + (double)(excl + sum) >= target) {
          uint64_t cum = excl;
          int q = 0;
          while (q < BPT - 1 && (double)before + (double)(cum + hv[q]) < target) cum += hv[q++];
          mine = i0 + q;
          s.bc_q[1] = cum;
        }
        const int sbb = blk_min_i(mine, s);
        const uint64_t before2 = before + s.bc_q[1];
        __syncthreads();
        if (sbb != 0x7fffffff) {
          // per chunk: the mass of bucket bb's sub-buckets below sbb (kept whatever the cut)
          if (t < P) s.cm[t] = rec[t * REC_WORDS + 3];
          __syncthreads();
          for (int f = t; f < P * sbb; f += CT) {
            const int c = f / sbb, i = f - c * sbb;
            const uint64_t v = a.stg[(row * P + c) * (int64_t)SSTRIDE + SCAP + i];
            if (v) atomicAdd(reinterpret_cast<unsigned long long*>(&s.cm[c]), (unsigned long long)v);
          }
          int lastp = -1;
          for (int c = 0; c < P; ++c) lastp = max(lastp, (int)(uint32_t)rec[c * REC_WORDS + 4]);
          if (t == 0) s.n_list = 0;
          __syncthreads();
          uint64_t* ent = r_gstage;
          auto take = [&](float z, int pos) __attribute__((always_inline)) {
            const int sb = gp_dsub(z, m, bb);
            if (sb < sbb) {
              if (mass_of(z, m) > 0) lastp = max(lastp, pos);
            } else if (sb == sbb) {
              const int i = atomicAdd(&s.n_list, 1);
              if (i < GKCAP2) ent[i] = ((uint64_t)f2key(z) << 32) | (uint32_t)pos;
            }
          };
          if (staged_all) {
            // the bucket's values are in the chunks' staging: no pass over the row
            for (int c = 0; c < P; ++c) {
              const uint64_t* src = a.stg + (row * P + c) * (int64_t)SSTRIDE;
              for (int i = t; i < s.cnt[c]; i += CT) {
                const uint64_t e = src[i];
                take(key2f((uint32_t)(e >> 32)), (int)(uint32_t)e);
              }
            }
          } else {
            bool sub_staged = true;  // k_gen_s staged the sub-bucket's values in every chunk
            int n_sub = 0;
            for (int c = 0; c < P; ++c) {
              const uint64_t w5 = rec[c * REC_WORDS + 5];
              const int nc = w5 ? (int)(w5 - 1) : -1;
              if (nc < 0 || nc > SCAP) sub_staged = false;
              else n_sub += nc;
            }
            if (sub_staged && n_sub <= GKCAP2) {
              for (int c = 0; c < P; ++c) lastp = max(lastp, (int)(uint32_t)rec[c * REC_WORDS + 6]);
              if (t == 0) {
                int off = 0;
                for (int c = 0; c < P; ++c) {
                  s.cut[c] = off;
                  off += (int)(rec[c * REC_WORDS + 5] - 1);
                }
                s.n_list = off;
              }
              __syncthreads();
              for (int c = 0; c < P; ++c) {
                const uint64_t* src = a.stg + (row * P + c) * (int64_t)SSTRIDE;
                const int nc = (int)(rec[c * REC_WORDS + 5] - 1);
                for (int i = t; i < nc; i += CT) ent[s.cut[c] + i] = src[i];
              }
            } else {
              // one pass over the row: a comparison per value, masses only inside bucket bb
              history_to_lds();
              for (int c = 0; c < P; ++c) {
                for_chunk<DT, SEG>(a, R, s, c, [&](float z, int pos) __attribute__((always_inline)) {
                  if (z > -INFINITY && z >= lo && gp_dbucket(z, m) == bb) take(z, pos);
                });
              }
            }
          }
          __syncthreads();
          const int n2 = s.n_list;
          __syncthreads();
          if (n2 <= GKCAP2) {
            const uint32_t kk = gp_topp_key(StagedPairs{ent, n2}, s, s.c.gen, lo, m, target, (double)before2);
            if (kk) {
              tau = fmaxf(lo, key2f(kk));
              for (int i = t; i < n2; i += CT) {
                const uint64_t e = ent[i];
                const float z = key2f((uint32_t)(e >> 32));
                if (z >= tau) {
                  const int pos = (int)(uint32_t)e;
                  const uint64_t w = mass_of(z, m);
                  atomicAdd(reinterpret_cast<unsigned long long*>(&s.cm[chunk_of(a, R, DT::VEC, pos)]),
                            (unsigned long long)w);
                  if (w > 0) lastp = max(lastp, pos);
                }
              }
              last = blk_max_i(lastp, s);  // its barriers also publish cm
              fast = true;
            }
          }
        }
      }
    }
  }
  float zid = -INFINITY;
  int id;
  if (fast) {
    id = gp_draw<DT, SEG>(a, R, s, tau, m, d.u, &zid, true, last);
  } else {
    // the crossing sub-bucket did not fit the staging: the single-workgroup nucleus selection
    history_to_lds();
    bool fused = gp_topp_fused<DT, SEG>(a, R, s, lo, m, (double)d.p, tau, last);
    if (!fused) {
      const uint32_t kk = gp_topp<DT, SEG>(a, R, s, lo, m, (double)d.p);
      tau = kk ? fmaxf(lo, key2f(kk)) : lo;
    }
    id = gp_draw<DT, SEG>(a, R, s, tau, m, d.u, &zid, fused, last);
  }
  // leave the workspace as it was found
  __syncthreads();
  if (d.topp) {
    uint64_t* lbase = a.lists + (row * P) * (int64_t)LCAPC;
    for (int i = t; i < P * LCAPC; i += CT) lbase[i] = 0;
    for (int c = 0; c < P; ++c) {
      const uint64_t w2 = rec[c * REC_WORDS + 2];
      const uint64_t w5 = rec[c * REC_WORDS + 5];
      const int nc = max(w2 ? min((int)(w2 - 1), SCAP) : 0, w5 ? min((int)(w5 - 1), SCAP) : 0);
      uint64_t* sb = a.stg + (row * P + c) * (int64_t)SSTRIDE;
      for (int i = t; i < nc; i += CT) sb[i] = 0;
      if (w2) for (int i = t; i < GDB; i += CT) sb[SCAP + i] = 0;
    }
  }
  __syncthreads();
  uint64_t* rw = a.rec + (row * P) * (int64_t)REC_WORDS;
  for (int i = t; i < P * REC_WORDS; i += CT) rw[i] = 0;
  if (t < RS_WORDS) a.rstate[row * RS_WORDS + t] = 0;
  if (t == 0) {
    a.out_ids[row] = id;
    a.out_logprobs[row] = id >= 0 ? (float)((double)zid - (double)m - d.L) : -INFINITY;
    if (a.next_tokens) {
      const int32_t dst = a.backfill_dest[row];
      if (dst >= 0 && (int64_t)dst < a.next_len) a.next_tokens[dst] = id;
    }
  }
}

// The deferred-row launches take the resolution kernel's list of deferred rows (dq[0] rows, their
// indices from dq[2]): at most GEN_GRID workgroups walk the (row, chunk) items and at most GEN_ROWS the
// rows, so that a call with no deferred row costs one small grid per launch (the two sizes measured
// best on rows of 152064 and 256000 logits).  The workgroups of k_gen_c that take a row count their
// arrivals in dq[1], and the last of them zeroes the list once all of them have read it; the others
// do nothing whether they read dq[0] before or after it is zeroed, so a call without deferred rows
// makes no atomic on the counter (one contended counter cost every workgroup a few microseconds).
constexpr int GEN_GRID = 1024;
constexpr int GEN_ROWS = 512;

template <class DT, bool SEG, int K>
__device__ __forceinline__ void gen_chunks(const SArgs& a, SSm& s) {
  const int64_t n = (int64_t)a.dq[0] * a.P;
  for (int64_t item = blockIdx.x; item < n; item += gridDim.x) {
    const int64_t row = a.dq[2 + item / a.P];
    const int c = (int)(item % a.P);
    if (K == 0) gen_a_item<DT, SEG>(a, s, row, c);
    else if (K == 1) gen_b_item<DT, SEG>(a, s, row, c);
    else gen_s_item<DT, SEG>(a, s, row, c);
    __syncthreads();  // the next item reuses the LDS
  }
}

template <class DT, bool SEG>
__global__ __launch_bounds__(CT) void k_gen_a(SArgs a) {
  __shared__ SSm s;
  gen_chunks<DT, SEG, 0>(a, s);
}
template <class DT, bool SEG>
__global__ __launch_bounds__(CT) void k_gen_b(SArgs a) {
  __shared__ SSm s;
  gen_chunks<DT, SEG, 1>(a, s);
}
template <class DT, bool SEG>
__global__ __launch_bounds__(CT) void k_gen_s(SArgs a) {
  __shared__ SSm s;
  gen_chunks<DT, SEG, 2>(a, s);
}

template <class DT, bool SEG>
__global__ __launch_bounds__(CT, 1) void k_gen_c(SArgs a) {
  __shared__ SSm s;
  const int n = a.dq[0];
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    gen_c_item<DT, SEG>(a, s, a.dq[2 + i]);
    __syncthreads();
  }
  const unsigned working = (unsigned)min(n, (int)gridDim.x);
  if (threadIdx.x == 0 && blockIdx.x < working) {
    if (atomicAdd(reinterpret_cast<unsigned int*>(&a.dq[1]), 1u) == working - 1) {
      for (int i = 0; i < n; ++i) a.dq[2 + i] = 0;
      a.dq[0] = 0;
      a.dq[1] = 0;
    }
  }
}

// ----------------------------------------------------------------------------------------------
// The kernel: one workgroup per (row, chunk)
// ----------------------------------------------------------------------------------------------
template <class DT, bool SEG>
__global__ __launch_bounds__(CT, 4) void k_stream(SArgs a) {
  __shared__ SSm s;
  const int t = threadIdx.x;
  constexpr int VEC = DT::VEC;
  int64_t L = blockIdx.x;
  if (a.xcd_map) L = (L & 7) * (a.grid >> 3) + (L >> 3);
  const int64_t row = L / a.P;
  const int c = (int)(L - row * a.P);
  SRow R;
  row_setup<DT, SEG>(a, row, c, R);

  // ---- the row's history first (HPT ids per thread, in registers): waiting for these loads then
  //      never waits for the row data issued after them (the vector memory counter is in order) ----
  // Loads are unconditional (indices clamped into range, or a dummy address when there is nothing to
  // read: the workspace's first bytes, always valid) so that none waits for another -- a load under a
  // branch is followed by a wait for it before the branch closes.
  const void* dummy = a.rec;
  constexpr int HPT = 16;
  int32_t hreg[HPT];
  const int nh = R.pen_on ? (int)min(R.h_hi - R.h_lo, (int64_t)HPT * CT) : 0;  // ids held in hreg
  {
    const int32_t* hrow = nh > 0 ? a.prm.hist_ids + R.h_lo : static_cast<const int32_t*>(dummy);
    static_for<HPT>([&](auto Q) {
      constexpr int q = decltype(Q)::value;
      hreg[q] = hrow[min(t + q * CT, max(nh - 1, 0))];
    });
  }
  // A penalised row's history arrives before its row data is requested: with every workgroup's row
  // loads in flight the history would wait behind them, and the overlay (hence the pass) with it.
  if (R.pen_on) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  asm volatile("" ::: "memory");  // the row loads stay behind the history loads

  // ---- the chunk's slots: one 16-byte non-temporal load each; the first LA are issued here, slot
  //      j + LA just before slot j is processed, so a wave whose issue stalls on a full memory queue
  //      still has arrived slots to work on ----
  const int ns = (int)(R.s1 - R.s0);  // body slots of the chunk; slot j of thread t is j * CT + t
  constexpr int LA = 8;
  uint4 d[CJ];
  auto issue = [&](auto J) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    const uint4* sp = ns > 0 ? slot_ptr<DT, SEG>(a, R, R.s0 + min(j * CT + t, ns - 1)) : static_cast<const uint4*>(dummy);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(sp));
    d[j] = make_uint4(v.x, v.y, v.z, v.w);
  };
  static_for<CJ>([&](auto J) {
    if constexpr (decltype(J)::value < LA) issue(J);
  });

  if (t < HXN) s.hx_pos[t] = -1;
  if (t == 0) {
    s.n_list = 0;
    s.flags = 0;
    s.hst_on = 0;
  }

  // ---- penalty overlay of the chunk's range ----
  const int64_t e_base = (int64_t)R.head + (R.s0 - 1) * VEC;  // row position of bitmap bit 0
  const int nwords = (int)(((R.s1 - R.s0 + 2) * VEC + 31) >> 5);
  int n_x = 0;  // penalised extras
  uint32_t tfl = 0;
  if (R.pen_on) n_x = build_overlay<HPT>(a, R, s, c, R.s0, R.s1, VEC, hreg, &tfl);
  if (tfl) atomicOr(&s.flags, tfl);

  // ---- one pass over the slots in arrival order: the penalised elements leave the registers for
  //      the extras, then the slot's maximum and its exponentials against a running reference
  //      (moved to each new thread maximum, with the sum rescaled), so the pass keeps pace with the
  //      loads instead of waiting for the whole chunk ----
  const float r = R.r;
  float xref = -INFINITY;       // running maximum of x
  float mref_t = MREF0;         // fl32(fl32(xref r) L2E), the exponent reference
  float acc0 = 0.0f, acc1 = 0.0f;
  int jbest = -1;  // the slot where the thread's body maximum was first reached
  // the overlay word of a slot (and its word prefix), read one slot ahead so that the LDS latency
  // hides behind the previous slot's arithmetic
  const int last_slot = max(ns - 1, 0);
  auto ov_bit0 = [&](int j) __attribute__((always_inline)) { return (min(j * CT + t, last_slot) + 1) * VEC; };
  uint32_t ov_word = 0, ov_pref = 0;
  if (R.pen_on) {
    ov_word = s.c.p.bitmap[ov_bit0(0) >> 5];
    ov_pref = s.c.p.wpref[ov_bit0(0) >> 5];
  }
  static_for<CJ>([&](auto J) {
    constexpr int j = decltype(J)::value;
    if constexpr (j + LA < CJ) issue(std::integral_constant<int, j + LA>{});
    const uint32_t word = ov_word, wpre = ov_pref;
    if constexpr (j + 1 < CJ) {
      if (R.pen_on) {
        ov_word = s.c.p.bitmap[ov_bit0(j + 1) >> 5];
        ov_pref = s.c.p.wpref[ov_bit0(j + 1) >> 5];
      }
    }
    {  // slot j is processed here and not earlier: no slot's values are hoisted into registers
      uint32_t x0 = d[j].x, x1 = d[j].y, x2 = d[j].z, x3 = d[j].w;
      asm volatile("" : "+v"(x0), "+v"(x1), "+v"(x2), "+v"(x3));
      d[j] = make_uint4(x0, x1, x2, x3);
    }
    if ((j + 1) * CT > ns && j * CT + t >= ns) d[j] = make_uint4(DT::NEG, DT::NEG, DT::NEG, DT::NEG);
    if (R.pen_on) {
      if (j * CT + t < ns) {
        // a slot's marked positions have consecutive numbers: stage their loaded values (their new
        // values are computed after the pass, one number per thread), mask them out of the registers
        const int b0 = (j * CT + t + 1) * VEC;
        const uint32_t bits = (word >> (b0 & 31)) & ((1u << VEC) - 1u);
        if (bits) {
          int rk = (int)wpre + __popc(word & ((1u << (b0 & 31)) - 1u));
          uint32_t rest = bits, applied = 0;
          while (rest) {
            const int e = __builtin_ctz(rest);
            rest &= rest - 1u;
            if (rk < XCAP) {
              s.c.p.xorig[rk] = __float_as_uint(elem<DT>(d[j], e));
              applied |= 1u << e;
            }
            ++rk;
          }
          const uint4 mk = DT::mask_of(applied);
          d[j].x = (d[j].x & ~mk.x) | (DT::NEG & mk.x);
          d[j].y = (d[j].y & ~mk.y) | (DT::NEG & mk.y);
          d[j].z = (d[j].z & ~mk.z) | (DT::NEG & mk.z);
          d[j].w = (d[j].w & ~mk.w) | (DT::NEG & mk.w);
        }
      }
    }
    float v = elem<DT>(d[j], 0);
#pragma unroll
    for (int e = 1; e < VEC; ++e) v = fmaxf(v, elem<DT>(d[j], e));
    if (v > xref) {
      xref = v;
      jbest = j;
      const float mnew = __fmul_rn(__fmul_rn(v, r), L2E);
      const float sc = rel2(mref_t, mnew);
      acc0 *= sc;
      acc1 *= sc;
      mref_t = mnew;
    }
#pragma unroll
    for (int e = 0; e < VEC; e += 2) {
      acc0 += __builtin_amdgcn_exp2f(__builtin_fmaf(__fmul_rn(elem<DT>(d[j], e), r), L2E, -mref_t));
      acc1 += __builtin_amdgcn_exp2f(__builtin_fmaf(__fmul_rn(elem<DT>(d[j], e + 1), r), L2E, -mref_t));
    }
  });
  const float xbody = xref;  // the thread's maximum over its body slots (first reached in slot jbest)
  // the unaligned head (chunk 0) and tail (last chunk) positions
  {
    int pos = -1;
    if (c == 0 && t < R.head) pos = t;
    else if (c == R.P - 1 && t >= 8 && t < 8 + (R.V - R.tail_lo)) pos = R.tail_lo + (t - 8);
    if (pos >= 0) {
      const float x = load_elem<DT, SEG>(a, R, pos);
      bool pen = false;
      if (R.pen_on) {
        const int rank = overlay_rank(s, (int)(pos - e_base));
        if (rank >= 0) {
          s.c.p.xorig[rank] = __float_as_uint(x);
          pen = true;
        }
      }
      if (!pen) {
        s.hx_pos[t] = pos;
        s.hx_val[t] = x;
      }
    }
  }
  __syncthreads();
  // the extras this thread owns join its maximum and its sum
  const bool own_hx = t < HXN && s.hx_pos[t] >= 0;
  {
    float xe = -INFINITY;
    for (int i = t; i < n_x; i += CT) {
      const float v = penalise_cv(__uint_as_float(s.c.p.xorig[i]), s.c.p.xval[i], R.rep, R.freq, R.pres);
      s.c.p.xval[i] = __float_as_uint(v);
      xe = fmaxf(xe, v);
    }
    if (own_hx) xe = fmaxf(xe, s.hx_val[t]);
    if (xe > xref) {
      xref = xe;
      const float mnew = __fmul_rn(__fmul_rn(xe, r), L2E);
      const float sc = rel2(mref_t, mnew);
      acc0 *= sc;
      acc1 *= sc;
      mref_t = mnew;
    }
    for (int i = t; i < n_x; i += CT)
      acc0 += __builtin_amdgcn_exp2f(__builtin_fmaf(__fmul_rn(__uint_as_float(s.c.p.xval[i]), r), L2E, -mref_t));
    if (own_hx) acc1 += __builtin_amdgcn_exp2f(__builtin_fmaf(__fmul_rn(s.hx_val[t], r), L2E, -mref_t));
  }
  const float zt = canon(xref, r);
  const float st = acc0 + acc1;

  // ---- chunk totals: waves on DPP, then the four waves in order ----
  {
    const float Mw = wave_max(mref_t);
    const float Sw = wave_sum(st * rel2(mref_t, Mw));
    const float Zw = wave_max(zt);
    if (lane_id() == 0) {
      s.wred[0][wave_id()] = Mw;
      s.wred[1][wave_id()] = Sw;
      s.wred[2][wave_id()] = Zw;
    }
  }
  __syncthreads();
  float cm = s.wred[0][0], cs = s.wred[1][0], zmax = s.wred[2][0];
  for (int w = 1; w < CW; ++w) {
    lse_add(cm, cs, s.wred[0][w], s.wred[1][w]);
    zmax = fmaxf(zmax, s.wred[2][w]);
  }
  uint32_t cflags = s.flags;
  bool has_fin = zmax > -INFINITY;
  if (!(zmax < INFINITY) || cs != cs) {
    // a NaN or +inf processed value: flag the row; whether any value is finite needs a look at each
    cflags |= FLAG_BAD_INPUT;
    uint32_t f = 0;
    reload_barrier(d);
    static_for<CJ>([&](auto J) {
      constexpr int j = decltype(J)::value;
#pragma unroll
      for (int e = 0; e < VEC; ++e) f |= isfinite(canon(elem<DT>(d[j], e), r)) ? 1u : 0u;
    });
    for (int i = t; i < n_x; i += CT) f |= isfinite(canon(__uint_as_float(s.c.p.xval[i]), r)) ? 1u : 0u;
    if (own_hx) f |= isfinite(canon(s.hx_val[t], r)) ? 1u : 0u;
    has_fin = blk_or(f, s) != 0;
  }
  reload_barrier(d);
  // ---- greedy rows: lowest position of the maximum ----
  int argpos = -1;
  if (R.greedy) {
    int best = 0x7fffffff;
    if (jbest >= 0 && canon(xbody, 1.0f) == zmax) {
      // the lowest body position of the maximum is in slot jbest (slots ascend in position with j)
      uint4 dd = d[0];
      static_for<CJ>([&](auto J) {
        constexpr int jj = decltype(J)::value;
        if (jj > 0 && jbest == jj) dd = d[jj];
      });
      int eb = VEC - 1;
#pragma unroll
      for (int e = VEC - 1; e >= 0; --e)
        if (elem<DT>(dd, e) == xbody) eb = e;
      best = R.head + (int)(R.s0 + jbest * CT + t) * VEC + eb;
    }
    for (int i = t; i < n_x; i += CT)
      if (canon(__uint_as_float(s.c.p.xval[i]), 1.0f) == zmax) best = min(best, pos_of_rank(s, nwords, e_base, i));
    if (own_hx && canon(s.hx_val[t], 1.0f) == zmax) best = min(best, s.hx_pos[t]);
    argpos = blk_min_i(best, s);
  }

  // ---- candidate bounds from the per-thread maxima ----
  const int Kk = R.kon ? R.k : 0, Kn = a.n_top;
  const bool s2b = !R.greedy && (R.kon || R.minp_on);
  const bool want_list = s2b || Kn > 0;
  float bound = INFINITY;
  float bk = -INFINITY, bn = -INFINITY;  // bounds of the chunk's K-th and n-th largest values
  if (want_list) {
    if (Kk > 0 || Kn > 0) {
      // Per wave, the R-th largest of its 64 thread maxima (R = ceil(K / 4)), by taking the wave's
      // maximum out R - 1 times (DPP reductions, no LDS); the smallest of the four waves' values
      // bounds the chunk's K-th largest value from below: each wave holds R values at least that
      // large, 4 R >= K in all.
      const int Rk = Kk > 0 ? (Kk + CW - 1) / CW : 0, Rn = Kn > 0 ? (Kn + CW - 1) / CW : 0;
      const int Rm = min(max(Rk, Rn), 64);
      const int l = lane_id();
      float v = zt, wk = -INFINITY, wn = -INFINITY;
      for (int it = 0; it < Rm; ++it) {
        const float mx = wave_max(v);
        if (it == Rk - 1) wk = mx;
        if (it == Rn - 1) wn = mx;
        const uint64_t hit = __ballot(v == mx);
        if (hit != 0 && l == (int)__builtin_ctzll(hit)) v = -INFINITY;
      }
      __syncthreads();  // every thread has read the chunk totals out of wred
      if (l == 0) {
        s.wred[0][wave_id()] = Rk <= 64 ? wk : -INFINITY;
        s.wred[1][wave_id()] = Rn <= 64 ? wn : -INFINITY;
      }
      __syncthreads();
      bk = fminf(fminf(s.wred[0][0], s.wred[0][1]), fminf(s.wred[0][2], s.wred[0][3]));
      bn = fminf(fminf(s.wred[1][0], s.wred[1][1]), fminf(s.wred[1][2], s.wred[1][3]));
    }
    if (s2b) {
      const float bm = R.minp_on ? __fadd_rn(zmax, (float)log((double)R.minp)) : -INFINITY;
      const float b2 = fmaxf(Kk > 0 ? bk : -INFINITY, bm);
      bound = Kn > 0 ? fminf(b2, bn) : b2;
    } else {
      bound = bn;
    }
  }

  reload_barrier(d);
  // ---- gather the candidates z >= bound ----
  uint64_t* glist = a.lists + L * (int64_t)LCAPC;
  int n_list = 0;
  bool overflow = false;  // the kept-set bound's candidates do not fit: the general path decides the kept set
  // when they do not, a second round gathers the candidates above the top-n bound alone, so that the
  // list still carries the chunk's top n
  float gb = bound;
  for (int round = 0; want_list && round < 2; ++round) {
    uint32_t pm = 0;
    static_for<CJ>([&](auto J) {
      constexpr int j = decltype(J)::value;
      float v = elem<DT>(d[j], 0);
#pragma unroll
      for (int e = 1; e < VEC; ++e) v = fmaxf(v, elem<DT>(d[j], e));
      if (v > -INFINITY && canon(v, r) >= gb) pm |= 1u << j;
    });
    reload_barrier(d);
    // the flagged slots of this thread, one LDS add per slot for the space of its candidates
    while (pm) {
      const int j = __builtin_ctz(pm);
      pm &= pm - 1u;
      const int p0 = R.head + (int)(R.s0 + j * CT + t) * VEC;
      // slot j through a select chain written in the kernel body, so that the register slots stay
      // registers (a helper taking the slots by reference would index them as memory)
      uint4 dd = d[0];
      static_for<CJ>([&](auto J) {
        constexpr int jj = decltype(J)::value;
        if (jj > 0 && j == jj) dd = d[jj];
      });
      uint32_t cb = 0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float z = canon(elem<DT>(dd, e), r);
        if (z > -INFINITY && z >= gb) cb |= 1u << e;
      }
      int idx = atomicAdd(&s.n_list, __popc(cb));
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        if ((cb >> e) & 1u) {
          if (idx < LCAPC) s.c.list[idx] = cand_key(canon(elem<DT>(dd, e), r), p0 + e);
          ++idx;
        }
      }
    }
    for (int i = t; i < n_x; i += CT) {
      const float z = canon(__uint_as_float(s.c.p.xval[i]), r);
      if (z > -INFINITY && z >= gb) {
        const int idx = atomicAdd(&s.n_list, 1);
        if (idx < LCAPC) s.c.list[idx] = cand_key(z, pos_of_rank(s, nwords, e_base, i));
      }
    }
    if (own_hx) {
      const float z = canon(s.hx_val[t], r);
      if (z > -INFINITY && z >= gb) {
        const int idx = atomicAdd(&s.n_list, 1);
        if (idx < LCAPC) s.c.list[idx] = cand_key(z, s.hx_pos[t]);
      }
    }
    __syncthreads();
    n_list = s.n_list;
    if (round == 1) break;
    overflow = n_list > LCAPC;
    if (!(overflow && Kn > 0 && bn > bound)) break;
    __syncthreads();  // every thread has read the count
    if (t == 0) s.n_list = 0;
    __syncthreads();
    gb = bn;
    reload_barrier(d);
  }
  const bool list_fits = want_list && n_list <= LCAPC;

  reload_barrier(d);
  // ---- publish the list, sorted in descending key order (rank by counting) ----
  float qk = -INFINITY, qn = -INFINITY;
  if (list_fits) {
    const int P = R.P;
    const int qki = Kk > 0 ? (Kk + P - 1) / P - 1 : -1;
    const int qni = Kn > 0 ? (Kn + P - 1) / P - 1 : -1;
    if (t == 0) {
      s.bc_f[0] = -INFINITY;
      s.bc_f[1] = -INFINITY;
    }
    __syncthreads();
    for (int i = t; i < n_list; i += CT) {
      const uint64_t key = s.c.list[i];
      const int rank = count_above(s.c.list, n_list, key);
      glist[rank] = key;
      if (rank == qki) s.bc_f[0] = cand_z(key);
      if (rank == qni) s.bc_f[1] = cand_z(key);
    }
    __syncthreads();
    qk = s.bc_f[0];
    qn = s.bc_f[1];
  } else if (want_list) {
    // too many candidates even above the top-n bound (ties): the top n exactly, slowly
    n_list = 0;
    if (Kn > 0) {
      uint64_t prev = ~0ull;
      for (int it = 0; it < Kn; ++it) {
        uint64_t best = 0;
        reload_barrier(d);
#pragma unroll 1
        for (int j = 0; j < CJ; ++j) {
          const int64_t slot = R.s0 + (int64_t)j * CT + t;
          if (slot >= R.s1) continue;
          uint4 dd = d[0];
          static_for<CJ>([&](auto J) {
            constexpr int jj = decltype(J)::value;
            if (jj > 0 && j == jj) dd = d[jj];
          });
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const float z = canon(elem<DT>(dd, e), r);
            if (z > -INFINITY && z == z) {
              const uint64_t key = cand_key(z, R.head + (int)slot * VEC + e);
              if (key < prev && key > best) best = key;
            }
          }
        }
        for (int i = t; i < n_x; i += CT) {
          const float z = canon(__uint_as_float(s.c.p.xval[i]), r);
          if (z > -INFINITY && z == z) {
            const uint64_t key = cand_key(z, pos_of_rank(s, nwords, e_base, i));
            if (key < prev && key > best) best = key;
          }
        }
        if (own_hx) {
          const float z = canon(s.hx_val[t], r);
          if (z > -INFINITY && z == z) {
            const uint64_t key = cand_key(z, s.hx_pos[t]);
            if (key < prev && key > best) best = key;
          }
        }
        best = blk_max_u64(best, s);
        if (best == 0) break;
        if (t == 0) glist[it] = best;
        prev = best;
        n_list = it + 1;
      }
      qn = -INFINITY;  // the top-n staging then takes the whole short list
    }
  }

  // ---- publish the chunk record (read by the resolution kernel, which the stream orders after this
  //      launch: the end of a launch makes its stores visible to the next one on every XCD) ----
  if (t == 0) {
    ChunkPub p;
    p.zmax = zmax;
    p.mref = cm;
    p.s = cs;
    p.flags = cflags | (has_fin ? PUB_FINITE : 0u) | (overflow ? PUB_OVER : 0u);
    p.argpos = argpos;
    p.n_list = n_list;
    p.qk = qk;
    p.qn = qn;
    rec_store(a.rec + L * REC_WORDS, p);
  }
}

// ----------------------------------------------------------------------------------------------
// The resolution kernel: one workgroup per row, after the chunk kernel
// ----------------------------------------------------------------------------------------------

template <class DT, bool SEG>
__global__ __launch_bounds__(CT, 1) void k_resolve(SArgs a) {
  __shared__ SSm s;
  const int t = threadIdx.x;
  SRow R;
  row_setup<DT, SEG>(a, (int64_t)blockIdx.x, 0, R);
  // the output history to LDS (all of a thread's loads in flight together) for the general path, which
  // groups it by chunk if the row needs it
  if (t == 0) s.hst_on = 0;
  const int64_t nh = R.h_hi - R.h_lo;
  if (R.pen_on && nh > 0 && nh <= HSTAGE) {
    constexpr int Q = HSTAGE / CT;
    int32_t v[Q];
    static_for<Q>([&](auto I) {
      constexpr int q = decltype(I)::value;
      v[q] = a.prm.hist_ids[R.h_lo + min((int64_t)(t + q * CT), nh - 1)];
    });
    static_for<Q>([&](auto I) {
      constexpr int q = decltype(I)::value;
      if (t + q * CT < nh) r_hstage[t + q * CT] = v[q];
    });
    if (t == 0) s.hst_on = 1;
  }
  __syncthreads();
  resolve_row<DT, SEG>(a, R, s);
}

// ----------------------------------------------------------------------------------------------
// Host side
// ----------------------------------------------------------------------------------------------
struct SGeo {
  int P;
  int64_t chunk_slots;
  bool ok;
};

SGeo geometry(int64_t B, int64_t V, albireo_dtype_t dtype) {
  SGeo g{0, 0, false};
  const int vec = dtype == ALBIREO_BF16 ? BF16T::VEC : F32T::VEC;
  const int64_t body = V / vec;
  int64_t P = (body + CSLOTS - 1) / CSLOTS;
  if (P < 1) P = 1;
  if (P > MAXPC || B <= 0 || B * P >= ((int64_t)1 << 31)) return g;
  g.P = (int)P;
  g.chunk_slots = (body + P - 1) / P;
  g.ok = true;
  return g;
}

struct WsParts {
  int64_t rec, lists, rstate, stg, dq, total;
};
WsParts ws_parts(int64_t B, int P) {
  WsParts w;
  w.rec = 0;
  w.lists = align256(w.rec + B * P * (int64_t)REC_WORDS * 8);
  w.rstate = align256(w.lists + B * P * (int64_t)LCAPC * 8);
  w.stg = align256(w.rstate + B * (int64_t)RS_WORDS * 8);
  w.dq = align256(w.stg + B * P * (int64_t)SSTRIDE * 8);
  w.total = align256(w.dq + (2 + B) * 4);
  return w;
}

}  // namespace

namespace albireo_stream {

bool supported(int64_t B, int64_t V, albireo_dtype_t dtype) { return geometry(B, V, dtype).ok; }

size_t workspace_bytes(int64_t B, int64_t V, albireo_dtype_t dtype) {
  const SGeo g = geometry(B, V, dtype);
  if (!g.ok) return 0;
  return (size_t)ws_parts(B, g.P).total;
}

albireo_status_t launch(const Request& q) {
  const SGeo g = geometry(q.B, q.V, q.dtype);
  if (!g.ok) return ALBIREO_E_UNSUPPORTED;
  SArgs a;
  memset(&a, 0, sizeof a);
  a.logits = static_cast<const unsigned char*>(q.logits);
  a.B = q.B;
  a.V = q.V;
  a.ld = q.ld;
  if (q.params) {
    const albireo_params_t* p = q.params;
    a.prm.temperature = p->temperature;
    a.prm.top_k = p->top_k;
    a.prm.top_p = p->top_p;
    a.prm.min_p = p->min_p;
    a.prm.rep = p->repetition_penalty;
    a.prm.freq = p->frequency_penalty;
    a.prm.pres = p->presence_penalty;
    a.prm.hist_offsets = p->hist_offsets;
    a.prm.hist_ids = p->hist_ids;
    a.prm.hist_len = p->hist_len;
    a.prompt_offsets = p->prompt_offsets;
    a.prompt_ids = p->prompt_ids;
    a.prompt_len = p->prompt_len;
    if (p->state) {
      a.st_ids = p->state->ids;
      a.st_counts = p->state->counts;
      a.st_len = p->state->len;
      a.st_flags = p->state->flags;
      a.st_cap = p->state->cap;
    }
  }
  a.uniforms = q.uniforms;
  a.out_ids = q.out_ids;
  a.out_logprobs = q.out_logprobs;
  a.n_top = q.n_top;
  a.out_top_ids = q.out_top_ids;
  a.out_top_logprobs = q.out_top_logprobs;
  a.out_flags = q.out_flags;
  if (q.step) {
    a.rng_on = 1;
    a.rng_seed = q.step->seed;
    a.rng_step = q.step->step;
    a.seq_ids = q.step->seq_ids;
    a.next_tokens = q.step->next_tokens;
    a.backfill_dest = q.step->backfill_dest;
    a.next_len = q.step->next_len;
  }
  const int es = q.dtype == ALBIREO_BF16 ? 2 : 4;
  if (q.shards) {
    const int64_t Ls = q.shards->shard_len, Ss = q.shards->shard_stride;
    const int64_t t = (q.V + Ls - 1) / Ls;
    const int64_t sps = Ls * es / 16;
    a.seg_sps = (uint32_t)sps;
    a.seg_magic = (uint32_t)(0xffffffffull / (uint64_t)sps);
    a.seg_gap = t > 1 ? (Ss - Ls) * es : 0;
  }
  a.P = g.P;
  a.chunk_slots = g.chunk_slots;
  a.grid = q.B * g.P;
  a.xcd_map = (a.grid % 8 == 0) ? 1 : 0;
  const WsParts w = ws_parts(q.B, g.P);
  a.rec = reinterpret_cast<uint64_t*>(q.ws + w.rec);
  a.lists = reinterpret_cast<uint64_t*>(q.ws + w.lists);
  a.rstate = reinterpret_cast<uint64_t*>(q.ws + w.rstate);
  a.stg = reinterpret_cast<uint64_t*>(q.ws + w.stg);
  a.dq = reinterpret_cast<int32_t*>(q.ws + w.dq);
  void* args[] = {&a};
  const void *fc, *fr, *ga, *gb, *gs, *gc;
#define ALBIREO_STREAM_KERNELS(DT)                                                                  \
  if (q.shards) {                                                                                   \
    fc = reinterpret_cast<const void*>(&k_stream<DT, true>);                                        \
    fr = reinterpret_cast<const void*>(&k_resolve<DT, true>);                                       \
    ga = reinterpret_cast<const void*>(&k_gen_a<DT, true>);                                         \
    gb = reinterpret_cast<const void*>(&k_gen_b<DT, true>);                                         \
    gs = reinterpret_cast<const void*>(&k_gen_s<DT, true>);                                         \
    gc = reinterpret_cast<const void*>(&k_gen_c<DT, true>);                                         \
  } else {                                                                                          \
    fc = reinterpret_cast<const void*>(&k_stream<DT, false>);                                       \
    fr = reinterpret_cast<const void*>(&k_resolve<DT, false>);                                      \
    ga = reinterpret_cast<const void*>(&k_gen_a<DT, false>);                                        \
    gb = reinterpret_cast<const void*>(&k_gen_b<DT, false>);                                        \
    gs = reinterpret_cast<const void*>(&k_gen_s<DT, false>);                                        \
    gc = reinterpret_cast<const void*>(&k_gen_c<DT, false>);                                        \
  }
  if (q.dtype == ALBIREO_BF16) {
    ALBIREO_STREAM_KERNELS(BF16T)
  } else {
    ALBIREO_STREAM_KERNELS(F32T)
  }
#undef ALBIREO_STREAM_KERNELS
  // chunk pass, row resolution, then the deferred rows' chunk-parallel general path
  hipError_t e = hipLaunchKernel(fc, dim3((unsigned)a.grid), dim3(CT), args, 0, q.stream);
  if (e == hipSuccess) e = hipLaunchKernel(fr, dim3((unsigned)q.B), dim3(CT), args, 0, q.stream);
  const unsigned gg = (unsigned)min(a.grid, (int64_t)GEN_GRID), gr = (unsigned)min(q.B, (int64_t)GEN_ROWS);
  if (e == hipSuccess) e = hipLaunchKernel(ga, dim3(gg), dim3(CT), args, 0, q.stream);
  if (e == hipSuccess) e = hipLaunchKernel(gb, dim3(gg), dim3(CT), args, 0, q.stream);
  if (e == hipSuccess) e = hipLaunchKernel(gs, dim3(gg), dim3(CT), args, 0, q.stream);
  if (e == hipSuccess) e = hipLaunchKernel(gc, dim3(gr), dim3(CT), args, 0, q.stream);
  return e == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

}  // namespace albireo_stream
