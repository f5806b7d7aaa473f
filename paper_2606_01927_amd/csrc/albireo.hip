// albireo.hip -- the register-resident sampling kernels, the standalone helpers and the C ABI of the
// per-sequence sampling library.
//
// k_sample: one 512-thread workgroup per row keeps the whole row in VGPRs (up to 38 16-byte slots per
// thread: bf16 rows up to 155655 logits, fp32 up to 77827).  Every logit is read from HBM once with
// 16-byte loads issued up front.  On that resident data the workgroup runs
//   * the penalty overlay (the feature list of sec. 8.1): the row's history ids mark a per-slot LDS
//     presence bitmap, the marked entries are masked in the registers and their new values live in a
//     small LDS "extras" list together with the few unaligned head/tail entries of the row;
//   * an online max / sum-exp pass overlapped with the loads, giving the full-vocabulary log-sum-exp
//     the logprobs need (sec. 2.1; App. A returns the sampled id with its probability);
//   * a candidate gather above a provable lower bound of the kept set (the K-th largest per-thread
//     maximum for top-k / top-n, m + ln(min_p) for min-p);
//   * exact resolution of top-k / min-p / top-p and the inverse-CDF draw on that small LDS list or,
//     when the kept set has no small bound, selections over distance buckets and a draw over re-reads
//     of the row.
// k_sample_multi: the same on P <= 8 chunk workgroups of a row in one cooperative launch (bounded waits
// through the caller's workspace); used by albireo_topk_topp on wide rows, and by sampling only for
// batches the streaming kernels cannot index.  Wider rows, and rows with a prompt history or a penalty
// state, go to the streaming kernels (stream.hip).  The choice is made by route_of, on the shape alone.
// Rows never interact, which is what lets the paper split sampling across ranks by rows (sec. 6.1,
// Eq. opt_sample).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <utility>

#include "albireo.h"
#include "stream.h"

namespace {

#include "common.h"

// ----------------------------------------------------------------------------------------------
// Geometry and capacities
// ----------------------------------------------------------------------------------------------
constexpr int NT = 512;           // threads per workgroup (2 waves per SIMD, 256 VGPRs each)
constexpr int NW = NT / 64;       // waves per workgroup
constexpr int JMAX = 38;          // 16-byte register slots per thread (152 VGPRs of row data)
// Instantiated slot counts: a chunk of n slots runs on the smallest J with n <= J * NT, so a
// single-chunk row of that kernel has more than (previous size) * NT slots (less one for the
// unaligned head) and every thread's first live_slots_min(J) slots are live.
constexpr int JSIZES[4] = {8, 16, 32, JMAX};
__host__ __device__ constexpr int live_slots_min(int J) {
  return J == JSIZES[3] ? JSIZES[2] : J == JSIZES[2] ? JSIZES[1] : J == JSIZES[1] ? JSIZES[0] : 0;
}
constexpr int UCAP = ALBIREO_MAX_UNIQUE_HISTORY;  // tracked distinct ids (history + head/tail)
constexpr int NWORDS = JMAX * NT / 4;             // presence bitmap words (one byte per register slot)
constexpr int LCAP = 2048;        // candidate list capacity
constexpr int EPT = LCAP / NT;    // list entries per thread in the list scans
constexpr int MAXP = 8;           // chunks per row supported
// Per-launch arguments (passed by value).
struct KArgs {
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
  float* out_probs;
  float* out_threshold;
  int32_t* out_kept;
  float* out_log_norm;
  // device random numbers: the uniform of a row from (seed, step, its sequence id) instead of uniforms
  int32_t rng_on;
  uint64_t rng_seed, rng_step;
  const int64_t* seq_ids;  // NULL: the row index
  // early-feedback backfill: the sampled id of row r also goes to next_tokens[backfill_dest[r]]
  int32_t* next_tokens;
  const int32_t* backfill_dest;
  int64_t next_len;
  // all-to-all receive layout: the row is split into blocks of seg_sps 16-byte slots, block b of row i
  // starting seg_gap bytes after the end of block b - 1 (the kernels built for it only)
  uint32_t seg_sps, seg_magic;  // slots per block; floor((2^32 - 1) / seg_sps)
  uint32_t seg_ntq, seg_ntr;    // NT = seg_ntq * seg_sps + seg_ntr
  int64_t seg_gap;
  int32_t mode;          // 0: sample, 1: topk_topp
  int32_t P;             // chunks per row
  int32_t n_groups;      // persistent row groups (grid = n_groups * P)
  int32_t xcd_map;       // place the P chunks of a group on one XCD
  int64_t chunk_slots;   // 16-byte body slots per chunk
  unsigned char* ws;
  int64_t ws_group_bytes;
};

// ----------------------------------------------------------------------------------------------
// Workspace layout of one row group (offsets 256-byte aligned)
// ----------------------------------------------------------------------------------------------
struct GroupSync {
  uint32_t arrive;
  uint32_t exit;
  uint32_t error;
  uint32_t pad[61];
};
struct ChunkStats {  // published by every chunk workgroup of a row
  float xm;          // max of the products x r over the chunk
  float mref;        // reference of s (log2 units)
  float s;           // sum of 2^(z*L2E - mref)
  uint32_t flags;
  float beta_sel;    // K-th largest per-thread maximum z of the chunk
  int32_t n_list;    // candidates gathered
  int32_t overflow;
  float w_total;     // general draw: chunk total
  int32_t last_pos;  // general draw: last position with positive weight / greedy argmax
  int32_t n_keep;    // general path: kept count
  float zmin;        // general path: min z over kept
  int32_t best;      // general path: lowest position of the maximum
  uint64_t zs_fix;   // general path: fixed-point mass of the kept set
  uint32_t pad[2];
};
struct GroupRes {    // published by the leader for the dense output
  float tau;
  float zs;
  int32_t id;
  int32_t pad[13];
};


struct WsLayout {
  int64_t sync, stats, res, hist, lists, total;
  __host__ __device__ WsLayout(int P) {
    sync = 0;
    stats = align256(sync + (int64_t)sizeof(GroupSync));
    res = align256(stats + (int64_t)sizeof(ChunkStats) * P);
    hist = align256(res + (int64_t)sizeof(GroupRes));
    lists = align256(hist + (int64_t)P * 256 * 8);
    total = align256(lists + (int64_t)P * LCAP * 8);
  }
};

struct Smem {
  alignas(16) uint32_t bitmap[NWORDS];  // one byte per body slot of the chunk, bit e = element e
  alignas(16) uint16_t wpref[NWORDS];   // set bits in the bitmap words before each word
  alignas(16) uint4 masktab[256];
  alignas(16) uint32_t x_cnt[UCAP];     // history count of each extras entry
  // per register slot and thread, the top 16 bits of the ordered key of the slot maximum (two slots
  // per word, slot-pair major): the gather's first pass reads these instead of the registers
  alignas(16) uint32_t scode[(JMAX + 1) / 2 * NT];
  int32_t x_pos[UCAP];             // extras: penalised body entries and head/tail entries
  float x_val[UCAP];
  uint64_t sk[LCAP];               // candidate list / sort keys
  float l_z[LCAP];                 // resolved list: z, weight, position in descending order
  float l_w[LCAP];
  int32_t l_p[LCAP];
  uint64_t hist[256];
  float red_f[2 * NW];
  uint32_t red_u[NW];
  uint64_t red_q[NW];
  int32_t n_body;  // extras entries of penalised body elements (position order); head/tail ones follow
  int32_t n_ext;   // all extras entries
  int32_t n_list;
  uint32_t flags;
  uint32_t ready;  // the row's penalty bitmap and hash are initialised (set by wave 0)
  alignas(16) float wp[6][NW];       // per-wave partials of the workgroup reduction
  alignas(16) uint32_t kh_cnt[256];  // K-th bound histogram: counts and minimum key per bucket
  alignas(16) uint32_t kh_min[256];
  uint64_t fxsum;                    // fixed-point mass of the extras
  int32_t bc_i[4];
  float bc_f[4];
  uint64_t bc_q[4];
  uint16_t first_u[4 * NT];  // extras entry of a thread's first occurrence of an id in the early
                             // count, or 0xffff
};
static_assert(sizeof(Smem) <= 160 * 1024, "LDS of one workgroup exceeds a gfx950 CU");
static_assert(64 * 32 <= UCAP, "history staging does not fit the extras arrays");


__device__ __forceinline__ float block_max(float v, Smem& s) {
  v = wave_max(v);
  __syncthreads();
  if (lane_id() == 0) s.red_f[wave_id()] = v;
  __syncthreads();
  float r = s.red_f[0];
  for (int w = 1; w < NW; ++w) r = fmaxf(r, s.red_f[w]);
  return r;
}
__device__ __forceinline__ float block_min(float v, Smem& s) { return -block_max(-v, s); }
__device__ __forceinline__ int block_min_i(int v, Smem& s) {
  v = wave_min_i(v);
  __syncthreads();
  if (lane_id() == 0) s.red_u[wave_id()] = (uint32_t)v;
  __syncthreads();
  int r = (int)s.red_u[0];
  for (int w = 1; w < NW; ++w) r = min(r, (int)s.red_u[w]);
  return r;
}
__device__ __forceinline__ int block_max_i(int v, Smem& s) {
  v = wave_max_i(v);
  __syncthreads();
  if (lane_id() == 0) s.red_u[wave_id()] = (uint32_t)v;
  __syncthreads();
  int r = (int)s.red_u[0];
  for (int w = 1; w < NW; ++w) r = max(r, (int)s.red_u[w]);
  return r;
}
__device__ __forceinline__ int block_sum_i(int v, Smem& s) {
  v = wave_sum_i(v);
  __syncthreads();
  if (lane_id() == 0) s.red_u[wave_id()] = (uint32_t)v;
  __syncthreads();
  int r = 0;
  for (int w = 0; w < NW; ++w) r += (int)s.red_u[w];
  return r;
}
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, Smem& s) {
  v = wave_sum_u64(v);
  __syncthreads();
  if (lane_id() == 0) s.red_q[wave_id()] = v;
  __syncthreads();
  uint64_t r = 0;
  for (int w = 0; w < NW; ++w) r += s.red_q[w];
  return r;
}
// (mref, s) pairs: s is relative to 2^mref
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  s = s * rel2(m, M) + s2 * rel2(m2, M);
  m = M;
}

// Exclusive scan over the NT threads in thread order.  *total is the last thread's exclusive prefix
// plus its own value, i.e. exactly the value a thread-serial continuation of the scan would give.
__device__ __forceinline__ float block_excl_scan(float v, Smem& s, float* total) {
  const int l = lane_id();
  const float incl = wave_incl_scan(v);
  const float excl = __uint_as_float(dpp_mov<DPP_WAVE_SHR1>(0u, __float_as_uint(incl)));
  __syncthreads();
  if (l == 63) s.red_f[wave_id()] = incl;
  __syncthreads();
  float off = 0.0f;
  for (int w = 0; w < wave_id(); ++w) off += s.red_f[w];
  const float e = off + excl;
  if (threadIdx.x == NT - 1) s.bc_f[3] = e + v;
  __syncthreads();
  *total = s.bc_f[3];
  __syncthreads();
  return e;
}


// ----------------------------------------------------------------------------------------------
// Row-group synchronisation through the workspace (P > 1).  The wait is bounded: after SPIN_LIMIT
// polls it records an error in the group's sync block and continues, so a bug cannot hang the GPU.
// The leader ORs FLAG_TIMEOUT into the flags of every row it writes once the error is set, and the
// group's last workgroup to exit clears it with the counters.
// ----------------------------------------------------------------------------------------------
__device__ __forceinline__ void group_barrier(GroupSync* gs, int P) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(&gs->arrive, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t target = (old / (uint32_t)P + 1u) * (uint32_t)P;
    uint32_t spins = 0;
    while ((int32_t)(__hip_atomic_load(&gs->arrive, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) - target) < 0) {
      __builtin_amdgcn_s_sleep(2);
      if (++spins > SPIN_LIMIT) {
        __hip_atomic_fetch_or(&gs->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  __syncthreads();
}

// ----------------------------------------------------------------------------------------------
// Bitonic sort of s.sk[0, npad) (npad a power of two <= LCAP)
// ----------------------------------------------------------------------------------------------
__device__ void bitonic_sort(Smem& s, int npad, bool descending) {
  __syncthreads();
  for (int size = 2; size <= npad; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < (npad >> 1); i += NT) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0) != descending;
        const uint64_t x = s.sk[lo], y = s.sk[hi];
        if ((x > y) == up) {
          s.sk[lo] = y;
          s.sk[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int next_pow2(int n) {
  int p = 2;
  while (p < n) p <<= 1;
  return p;
}

// ----------------------------------------------------------------------------------------------
// Per-row uniform state
// ----------------------------------------------------------------------------------------------
// fl32(log(min_p)), evaluated in double
__device__ __forceinline__ float log_minp_of(float minp) { return (float)log((double)minp); }

struct RowState {
  int64_t row;
  const unsigned char* rowp;
  int V;
  int head;            // elements before the first 16-byte boundary of the row
  int64_t body_slots;  // 16-byte slots after head
  int tail_lo;         // first element after the body
  int64_t s0, s1;      // this chunk's body slots [s0, s1)
  int c, P;
  bool owns_head, owns_tail;
  bool greedy;
  float r;             // temperature reciprocal
  int k;
  bool k_on, minp_on, topp_on;
  float p, minp;
  bool pen_on;
  float rep, freq, pres;
  int64_t h_lo, h_hi;
  float u;
  uint32_t flags;
  bool seg;            // the row is laid out in blocks (all-to-all receive layout)
  uint32_t sps, smagic;
  int64_t sgap;
};


// Block of a body slot in the blocked layout: the reciprocal-multiplier estimate is low by at most
// one for q < 2^31, which the remainder test corrects.
__device__ __forceinline__ uint32_t seg_of(const RowState& R, uint32_t q) {
  uint32_t g = __umulhi(q, R.smagic);
  if (q - g * R.sps >= R.sps) ++g;
  return g;
}
// Address of a row position (bytes), in either layout.
template <class DT>
__device__ __forceinline__ const unsigned char* pos_ptr(const RowState& R, int64_t pos) {
  const unsigned char* p = R.rowp + pos * DT::ES;
  if (R.seg) p += (int64_t)seg_of(R, (uint32_t)(pos / DT::VEC)) * R.sgap;
  return p;
}
template <class DT>
__device__ __forceinline__ float load_pos(const RowState& R, int64_t pos) {
  return DT::load1(pos_ptr<DT>(R, pos), 0);
}
// Byte offset of a body slot from the row's first element (the blocked layout has no head).
template <class DT>
__device__ __forceinline__ int64_t slot_off(const RowState& R, int64_t slot) {
  int64_t o = ((int64_t)R.head + slot * DT::VEC) * DT::ES;
  if (R.seg) o += (int64_t)seg_of(R, (uint32_t)slot) * R.sgap;
  return o;
}

// Row geometry from the kernel arguments alone (no loads), so the row loads can start at once.
template <class DT, bool SEG = false>
__device__ __forceinline__ void row_geometry(const KArgs& a, int64_t row, int c, RowState& R) {
  R.seg = SEG;
  R.sps = a.seg_sps;
  R.smagic = a.seg_magic;
  R.sgap = a.seg_gap;
  R.row = row;
  R.c = c;
  R.P = a.P;
  R.V = (int)a.V;
  R.rowp = a.logits + row * a.ld * DT::ES;
  const uint64_t addr = reinterpret_cast<uint64_t>(R.rowp);
  int head = (int)(((16u - (uint32_t)(addr & 15u)) & 15u) / DT::ES);
  if (head > R.V) head = R.V;
  R.head = head;
  R.body_slots = (R.V - head) / DT::VEC;
  R.tail_lo = head + (int)R.body_slots * DT::VEC;
  R.s0 = (int64_t)c * a.chunk_slots;
  if (R.s0 > R.body_slots) R.s0 = R.body_slots;
  R.s1 = R.s0 + a.chunk_slots;
  if (R.s1 > R.body_slots) R.s1 = R.body_slots;
  R.owns_head = (c == 0);
  R.owns_tail = (c == a.P - 1);
}

struct RawParams {
  float T, p, mp, rep, freq, pres, u;
  int k;
  int64_t lo, hi, seq;
};

// Issue the row's parameter loads (scalar, no branches); the values are used later, so the loads are
// in flight while the first row loads go out.
__device__ __forceinline__ RawParams row_params_load(const KArgs& a, int64_t row) {
  const DevParams& q = a.prm;
  RawParams rp;
  rp.T = sload(q.temperature ? q.temperature + row : &kParamDefaults[0]);
  rp.p = sload(q.top_p ? q.top_p + row : &kParamDefaults[1]);
  rp.mp = sload(q.min_p ? q.min_p + row : &kParamDefaults[2]);
  rp.rep = sload(q.rep ? q.rep + row : &kParamDefaults[3]);
  rp.freq = sload(q.freq ? q.freq + row : &kParamDefaults[4]);
  rp.pres = sload(q.pres ? q.pres + row : &kParamDefaults[5]);
  rp.u = sload(a.uniforms ? a.uniforms + row : &kParamDefaults[6]);
  rp.k = sload(q.top_k ? q.top_k + row : &kZeroI32[0]);
  const int64_t* ho = q.hist_offsets ? q.hist_offsets + row : &kZeroI64[0];
  rp.lo = sload(ho);
  rp.hi = sload(ho + 1);
  rp.seq = a.seq_ids ? sload(a.seq_ids + row) : row;
  return rp;
}

// Per-row parameters, with malformed values replaced by their "off" value and flagged.
__device__ __forceinline__ void row_params(const KArgs& a, RawParams rp, RowState& R) {
  uint32_t flags = 0;
  float T = rp.T, p = rp.p, mp = rp.mp, rep = rp.rep, freq = rp.freq, pres = rp.pres;
  const int k = rp.k;
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
  R.k_on = !R.greedy && k > 0 && (int64_t)k < a.V;
  R.minp_on = !R.greedy && mp > 0.0f;
  R.minp = mp > 1.0f ? 1.0f : mp;
  R.topp_on = !R.greedy && p < 1.0f;
  R.p = p;
  R.rep = rep;
  R.freq = freq;
  R.pres = pres;
  R.pen_on = false;
  R.h_lo = R.h_hi = 0;
  if (a.prm.hist_offsets) {
    const int64_t lo = rp.lo, hi = rp.hi;
    if (lo < 0 || hi < lo || hi > a.prm.hist_len) {
      flags |= FLAG_BAD_PARAM;
    } else if (hi > lo) {
      R.pen_on = true;
      R.h_lo = lo;
      R.h_hi = hi;
    }
  }
  R.u = a.rng_on ? philox_uniform(a.rng_seed, a.rng_step, (uint64_t)rp.seq) : rp.u;
  R.flags = flags;
}

typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));

// A thread's register slots of the chunk (16 bytes each), stored as register tuples of at most 32
// dwords -- 8-slot tuples, then a 4-slot and a 2-slot one -- so that a slot can also be read with a
// wave-uniform run-time index: inside one tuple that is a handful of indexed register moves, where
// an array of slots would need a chain of selects over every slot.
template <class DT, int J>
struct Chunk {
  static constexpr int NG = J / 8;             // 8-slot tuples
  static constexpr bool H4 = (J % 8) >= 4;     // a 4-slot tuple after them
  static constexpr bool H2 = (J % 4) >= 2;     // and a 2-slot tuple
  static_assert(J % 2 == 0 && NG <= 4, "unsupported slot count");
  u32x32 g[NG > 0 ? NG : 1];
  u32x16 h;
  u32x8 q;

  template <int j>
  __device__ __forceinline__ uint4 get() const {
    if constexpr (j < 8 * NG) {
      constexpr int o = 4 * (j % 8);
      return make_uint4(g[j / 8][o], g[j / 8][o + 1], g[j / 8][o + 2], g[j / 8][o + 3]);
    } else if constexpr (H4 && j < 8 * NG + 4) {
      constexpr int o = 4 * (j - 8 * NG);
      return make_uint4(h[o], h[o + 1], h[o + 2], h[o + 3]);
    } else {
      constexpr int o = 4 * (j - 8 * NG - (H4 ? 4 : 0));
      return make_uint4(q[o], q[o + 1], q[o + 2], q[o + 3]);
    }
  }
  template <int j>
  __device__ __forceinline__ void set(uint4 v) {
    if constexpr (j < 8 * NG) {
      constexpr int o = 4 * (j % 8);
      g[j / 8][o] = v.x;
      g[j / 8][o + 1] = v.y;
      g[j / 8][o + 2] = v.z;
      g[j / 8][o + 3] = v.w;
    } else if constexpr (H4 && j < 8 * NG + 4) {
      constexpr int o = 4 * (j - 8 * NG);
      h[o] = v.x;
      h[o + 1] = v.y;
      h[o + 2] = v.z;
      h[o + 3] = v.w;
    } else {
      constexpr int o = 4 * (j - 8 * NG - (H4 ? 4 : 0));
      q[o] = v.x;
      q[o + 1] = v.y;
      q[o + 2] = v.z;
      q[o + 3] = v.w;
    }
  }
  // slot j for a wave-uniform j in [0, J): a branch to its tuple, then indexed moves inside it
  __device__ __forceinline__ uint4 pick(int j) const {
    if (j < 8 * NG) {
      const int o = 4 * (j & 7);
      if (j < 8) return make_uint4(g[0][o], g[0][o + 1], g[0][o + 2], g[0][o + 3]);
      if constexpr (NG > 1) {
        if (j < 16) return make_uint4(g[1 % NG][o], g[1 % NG][o + 1], g[1 % NG][o + 2], g[1 % NG][o + 3]);
      }
      if constexpr (NG > 2) {
        if (j < 24) return make_uint4(g[2 % NG][o], g[2 % NG][o + 1], g[2 % NG][o + 2], g[2 % NG][o + 3]);
      }
      if constexpr (NG > 3) return make_uint4(g[3 % NG][o], g[3 % NG][o + 1], g[3 % NG][o + 2], g[3 % NG][o + 3]);
    }
    if constexpr (H4) {
      if (j < 8 * NG + 4) {
        const int o = 4 * (j - 8 * NG);
        return make_uint4(h[o], h[o + 1], h[o + 2], h[o + 3]);
      }
    }
    if constexpr (H2) {
      const int o = 4 * (j - 8 * NG - (H4 ? 4 : 0));
      return make_uint4(q[o], q[o + 1], q[o + 2], q[o + 3]);
    }
    return make_uint4(0u, 0u, 0u, 0u);
  }
};


// Double-precision per-row scalars, kept out of line so their polynomial constants never occupy
// registers of the streaming code.  Both are called where few registers are live: the first before any
// load of the row is issued, the second after the row's registers are released.
struct RowDoubles {
  double L;     // log sum_v exp(z_v - m)
  float zfull;  // sum_v exp(z_v - m)
};

// sum_v 2^(z_v L2E - mref) = S  =>  log sum_v e^(z_v - m) = ln S - D ln 2 with D = m L2E - mref (the
// exact offset of the reference, in double).
__device__ __noinline__ RowDoubles row_doubles(float mref, float S, float m) {
  RowDoubles o;
  const double D = (double)m * (double)L2E - (double)mref;
  o.L = log((double)S) - D * 0.6931471805599453;
  o.zfull = (float)exp(o.L);
  return o;
}

// Top-p candidate bound when top-p is the only filter: the elements below
// t0 = m + log((1 - p) Z / (2 V)) carry less than (1 - p) / 2 of the mass together, so the nucleus
// (whose complement below its last group holds at most 1 - p) lies at or above t0.  Evaluated in
// fp32 and lowered by a relative 1e-4, far more than the fp32 rounding of ln Z and of the sum.
__device__ __forceinline__ float topp_bound(float mref, float S, float m, float p, int V) {
  const float lnZ = __logf(S) - __builtin_fmaf(m, L2E, -mref) * 0.693147182f;
  const float t0 = m + lnZ + __logf((1.0f - p) * 0.5f / (float)V);
  return t0 - 1e-4f * (1.0f + fabsf(t0));
}

// ----------------------------------------------------------------------------------------------
// Per-row context shared by the resolution stages
// ----------------------------------------------------------------------------------------------
struct RowCtx {
  float m;         // max processed logit z of the row
  double L;        // log sum_v exp(z_v - m) over the full vocabulary
  float zfull;     // sum_v exp(z_v - m)
  float tau_m;     // min-p threshold (-inf when off)
  float row_beta;  // K-th largest per-thread maximum of the row
  int n_ext;       // extras in LDS
  int n_list;      // candidates in s.sk (at the leader: union over the chunks)
  GroupSync* gsync;
  ChunkStats* gstats;
  GroupRes* gres;
  uint64_t* ghist;
  uint64_t* glists;
};

// The outputs the out-of-line stages write, passed by value so the kernel arguments themselves never
// have their address taken (they stay in the kernarg segment and load through the scalar unit).
struct OutArgs {
  int32_t mode;
  int32_t n_top;
  int64_t V;
  int32_t* out_top_ids;
  float* out_top_logprobs;
  float* out_probs;
};

struct Resolution {
  float tau;    // kept set S = {finite z >= tau}
  float zs;     // sum over S of exp(z - m)
  float zmin;   // min z over S
  int kept;     // |S|
  int id;       // drawn (or greedy) token
  float zid;    // its processed logit
  int id_here;  // this workgroup writes out_ids / out_logprobs
};

// Iterate over the extras held in LDS (strided over threads).  BODY sees x and pos.
#define FOR_EXTRAS(S, NX, BODY)                                                                 \
  for (int xi_ = threadIdx.x; xi_ < (NX); xi_ += NT) {                                        \
    const float x = (S).x_val[xi_];                                                             \
    const int pos = (S).x_pos[xi_];                                                             \
    BODY                                                                                        \
  }

// Re-read one body slot of the chunk from memory with the penalised entries masked to -inf (their
// values are in the extras).  Used by the stages that run after the registers are released.
template <class DT>
__device__ __forceinline__ uint4 load_slot(const RowState& R, int64_t slot) {
  return *reinterpret_cast<const uint4*>(R.rowp + slot_off<DT>(R, slot));
}
// The penalised elements of a body slot read from memory set to -inf (their values are extras).
template <class DT>
__device__ __forceinline__ uint4 mask_slot(const RowState& R, const Smem& s, int64_t slot, uint4 d) {
  if (R.pen_on) {
    const int sl = (int)(slot - R.s0);
    const uint32_t byte = (s.bitmap[sl >> 2] >> ((sl & 3) * 8)) & 255u;
    const uint4 mk = s.masktab[byte];
    d.x = (d.x & ~mk.x) | (DT::NEG & mk.x);
    d.y = (d.y & ~mk.y) | (DT::NEG & mk.y);
    d.z = (d.z & ~mk.z) | (DT::NEG & mk.z);
    d.w = (d.w & ~mk.w) | (DT::NEG & mk.w);
  }
  return d;
}
template <class DT>
__device__ __forceinline__ uint4 load_masked(const RowState& R, const Smem& s, int64_t slot) {
  return mask_slot<DT>(R, s, slot, load_slot<DT>(R, slot));
}

// Iterate over the chunk's body elements re-read from memory.  BODY sees x and pos.  MEM_U slots per
// thread are loaded before any is used (unconditional loads: a slot past the chunk reloads the first
// of the group), so that one pass keeps MEM_U round trips in flight.
constexpr int MEM_U = 4;
#define FOR_MEM_ELEMS(R, S, BODY)                                                               \
  for (int64_t sb_ = (R).s0 + threadIdx.x; sb_ < (R).s1; sb_ += (int64_t)MEM_U * NT) {          \
    uint4 dd_[MEM_U];                                                                           \
    _Pragma("unroll") for (int u_ = 0; u_ < MEM_U; ++u_) {                                      \
      const int64_t sl_ = sb_ + (int64_t)u_ * NT;                                               \
      dd_[u_] = load_slot<DT>((R), sl_ < (R).s1 ? sl_ : sb_);                                   \
    }                                                                                           \
    _Pragma("unroll") for (int u_ = 0; u_ < MEM_U; ++u_) {                                      \
      const int64_t slot_ = sb_ + (int64_t)u_ * NT;                                             \
      if (slot_ < (R).s1) {                                                                     \
        const uint4 d_ = mask_slot<DT>((R), (S), slot_, dd_[u_]);                               \
        _Pragma("unroll") for (int e_ = 0; e_ < DT::VEC; ++e_) {                                \
          const float x = DT::get(d_, e_);                                                      \
          const int pos = (R).head + (int)slot_ * DT::VEC + e_;                                 \
          BODY                                                                                  \
        }                                                                                       \
      }                                                                                         \
    }                                                                                           \
  }

// Extras index of a row position in this chunk, or -1 when the position's value is in the registers
// (or belongs to another chunk).  Penalised body elements are numbered by their rank among the set
// bits of the presence bitmap (position order); the unaligned head / tail positions follow.
template <class DT>
__device__ __forceinline__ int extras_index(const Smem& s, const RowState& R, int pos) {
  if (pos < R.head) return R.owns_head ? s.n_body + pos : -1;
  if (pos >= R.tail_lo) return R.owns_tail ? s.n_body + (R.owns_head ? R.head : 0) + (pos - R.tail_lo) : -1;
  if (!R.pen_on) return -1;
  const int rel = pos - R.head;  // >= 0 here: a shift and a mask below
  const int sl = rel / DT::VEC - (int)R.s0;
  if ((unsigned)sl >= (unsigned)(R.s1 - R.s0)) return -1;
  const int b = (sl & 3) * 8 + rel % DT::VEC;
  const uint32_t word = s.bitmap[sl >> 2];
  if (!((word >> b) & 1u)) return -1;
  return (int)s.wpref[sl >> 2] + __popc(word & ((1u << b) - 1u));
}

// The processed-before-temperature value x of a row position: the extras value where the position has
// one, else the raw logit.
template <class DT>
__device__ __forceinline__ float x_at(const Smem& s, const RowState& R, int n_ext, int pos) {
  const int u = n_ext > 0 ? extras_index<DT>(s, R, pos) : -1;
  return u >= 0 ? s.x_val[u] : load_pos<DT>(R, pos);
}

// Gather the n_top-candidate list (or any list) above `bl` into s.sk; returns the count (may
// exceed LCAP, in which case the list is incomplete).
template <class DT>
__device__ int gather_mem(Smem& s, const RowState& R, int n_ext, float bl, bool strict) {
  __syncthreads();
  if (threadIdx.x == 0) s.n_list = 0;
  __syncthreads();
  const float r = R.r;
  FOR_MEM_ELEMS(R, s, {
    const float z = canon(x, r);
    if (z > -INFINITY && (strict ? z > bl : z >= bl)) {
      const int idx = atomicAdd(&s.n_list, 1);
      if (idx < LCAP) s.sk[idx] = cand_key(z, pos);
    }
  })
  FOR_EXTRAS(s, n_ext, {
    const float z = canon(x, r);
    if (z > -INFINITY && (strict ? z > bl : z >= bl)) {
      const int idx = atomicAdd(&s.n_list, 1);
      if (idx < LCAP) s.sk[idx] = cand_key(z, pos);
    }
  })
  __syncthreads();
  return s.n_list;
}

// Union of the chunk lists at the leader (P > 1).  Every chunk passes its own count; returns the
// total and whether any chunk (or the union) overflowed.  On return the leader holds the union in
// s.sk[0, total) when there is no overflow.
__device__ int union_lists(Smem& s, const RowState& R, const RowCtx& X, int n_own, bool& overflow) {
  const int P = R.P, c = R.c;
  if (threadIdx.x == 0) {
    st_agent(&X.gstats[c].n_list, (int32_t)n_own);
    st_agent(&X.gstats[c].overflow, (int32_t)overflow);
  }
  if (!overflow)
    for (int i = threadIdx.x; i < n_own; i += NT) st_agent(&X.glists[(int64_t)c * LCAP + i], s.sk[i]);
  group_barrier(X.gsync, P);
  int tot = 0;
  bool of = false;
  for (int q = 0; q < P; ++q) {
    tot += ld_agent(&X.gstats[q].n_list);
    of = of || ld_agent(&X.gstats[q].overflow) != 0;
  }
  overflow = of || tot > LCAP;
  if (!overflow && c == 0) {
    int off = 0;
    for (int q = 0; q < P; ++q) {
      const int nq = ld_agent(&X.gstats[q].n_list);
      if (q > 0)
        for (int i = threadIdx.x; i < nq; i += NT) s.sk[off + i] = ld_agent(&X.glists[(int64_t)q * LCAP + i]);
      off += nq;
    }
  }
  // every chunk has read the counts before any of them reuses the slots
  group_barrier(X.gsync, P);
  return tot;
}

// Sort s.sk[0, n) descending (z desc, position asc) and write the n_top outputs of the row.
__device__ void write_top_n(const OutArgs& a, Smem& s, const RowCtx& X, int64_t row, int n) {
  const int npad = next_pow2(n);
  for (int i = n + threadIdx.x; i < npad; i += NT) s.sk[i] = 0;
  bitonic_sort(s, npad, true);
  for (int t = threadIdx.x; t < a.n_top; t += NT) {
    const int64_t o = row * a.n_top + t;
    if (t < n) {
      a.out_top_ids[o] = cand_pos(s.sk[t]);
      a.out_top_logprobs[o] = (float)((double)cand_z(s.sk[t]) - (double)X.m - X.L);
    } else {
      a.out_top_ids[o] = -1;
      a.out_top_logprobs[o] = -INFINITY;
    }
  }
  __syncthreads();
}

// ----------------------------------------------------------------------------------------------
// Radix selection over the chunk (re-read from memory) and the extras (general path).
// Finds the largest key K such that the weight of eligible elements (finite z >= zlo) with
// key(z) >= K reaches the target; weights are counts (wmode 0) or fixed-point masses
// 2^32 * exp(z - m) (wmode 1).  A negative target means (-target) * (total eligible weight).
// Returns false when the target is not reached.  Uniform across the chunks of a row.
// ----------------------------------------------------------------------------------------------
template <class DT>
__device__ bool radix_select(Smem& s, const RowState& R, const RowCtx& X, float zlo, int wmode, double target,
                             uint32_t& out_key) {
  uint32_t prefix = 0;
  uint64_t above = 0;
  double tgt = target;
  const float r = R.r, m = X.m;
  const int P = R.P;
#pragma unroll 1
  for (int shift = 24; shift >= 0; shift -= 8) {
    __syncthreads();
    if (threadIdx.x < 256) s.hist[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t hi_mask = (shift == 24) ? 0u : (0xffffffffu << (shift + 8));
    FOR_MEM_ELEMS(R, s, {
      const float z = canon(x, r);
      if (z > -INFINITY && z >= zlo) {
        const uint32_t kz = f2key(z);
        if ((kz & hi_mask) == (prefix & hi_mask)) {
          const uint64_t wgt = wmode ? fixmass(__expf(z - m)) : 1ull;
          atomicAdd((unsigned long long*)&s.hist[(kz >> shift) & 255u], (unsigned long long)wgt);
        }
      }
    })
    FOR_EXTRAS(s, X.n_ext, {
      const float z = canon(x, r);
      if (z > -INFINITY && z >= zlo) {
        const uint32_t kz = f2key(z);
        if ((kz & hi_mask) == (prefix & hi_mask)) {
          const uint64_t wgt = wmode ? fixmass(__expf(z - m)) : 1ull;
          atomicAdd((unsigned long long*)&s.hist[(kz >> shift) & 255u], (unsigned long long)wgt);
        }
      }
    })
    __syncthreads();
    if (P > 1) {
      if (threadIdx.x < 256) st_agent(&X.ghist[(int64_t)R.c * 256 + threadIdx.x], s.hist[threadIdx.x]);
      group_barrier(X.gsync, P);
      uint64_t v = 0;
      if (threadIdx.x < 256)
        for (int q = 0; q < P; ++q) v += ld_agent(&X.ghist[(int64_t)q * 256 + threadIdx.x]);
      group_barrier(X.gsync, P);  // every chunk has read before anyone writes the next round
      if (threadIdx.x < 256) s.hist[threadIdx.x] = v;
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      if (tgt < 0) {  // the first round sees every eligible element: resolve the fractional target
        uint64_t tt = 0;
        for (int d = 0; d < 256; ++d) tt += s.hist[d];
        tgt = (double)tt * (-tgt);
      }
      uint64_t cum = above;
      int d = 255;
      for (; d >= 0; --d) {
        if ((double)(cum + s.hist[d]) >= tgt) break;
        cum += s.hist[d];
      }
      s.bc_i[0] = d;
      s.bc_q[0] = cum;
      s.bc_q[1] = (uint64_t)__double_as_longlong(tgt);
    }
    __syncthreads();
    const int d = s.bc_i[0];
    above = s.bc_q[0];
    tgt = __longlong_as_double((long long)s.bc_q[1]);
    __syncthreads();
    if (d < 0) return false;
    prefix |= (uint32_t)d << shift;
  }
  out_key = prefix;
  return true;
}

// Single-chunk rows: the selection radix_select makes (the key of the first group, in descending z,
// at which the cumulative count or fixed-point mass of the finite z >= zlo reaches the target; a
// negative target is that fraction of the total), with a first level over the distance from the row
// maximum instead of the top byte of the order key, whose few buckets collect most values and
// serialise the LDS atomics.  fl(m - z) scaled by SD_SCALE is monotone in z, so a lower bucket holds
// only larger values and equal values share a bucket.  The bucket where the cumulative crosses is
// staged in LDS and finished by the byte radix there, from the cumulative of the buckets above it; a
// bucket too large to stage (or a target of 0) goes to radix_select.
constexpr int SD_B = 2048;
constexpr float SD_SCALE = 64.0f;
constexpr int SD_CAP = 2 * LCAP;  // 32-bit keys in the 64-bit candidate list area
static_assert(sizeof(Smem::scode) >= SD_B * sizeof(uint64_t) && SD_B % NT == 0, "distance histogram does not fit");

__device__ __forceinline__ int dist_bucket(float z, float m) {
  const float d = __fmul_rn(__fsub_rn(m, z), SD_SCALE);
  return d < (float)(SD_B - 1) ? (int)d : SD_B - 1;
}

template <class DT>
__device__ bool select_dist(Smem& s, const RowState& R, const RowCtx& X, float zlo, int wmode, double target,
                            uint32_t& out_key) {
  const float r = R.r, m = X.m;
  uint64_t* h = reinterpret_cast<uint64_t*>(s.scode);
  uint32_t* keys = reinterpret_cast<uint32_t*>(s.sk);
  __syncthreads();
  for (int b = threadIdx.x; b < SD_B; b += NT) h[b] = 0;
  if (threadIdx.x == 0) {
    s.bc_i[0] = -1;
    s.bc_i[1] = 0;
  }
  __syncthreads();
  auto weight = [&](float z) __attribute__((always_inline)) -> uint64_t {
    return wmode ? fixmass(__expf(z - m)) : 1ull;
  };
  auto add = [&](float x) __attribute__((always_inline)) {
    const float z = canon(x, r);
    if (z > -INFINITY && z >= zlo)
      atomicAdd((unsigned long long*)&h[dist_bucket(z, m)], (unsigned long long)weight(z));
  };
  FOR_MEM_ELEMS(R, s, { add(x); })
  FOR_EXTRAS(s, X.n_ext, { add(x); })
  __syncthreads();
  // consecutive buckets per thread, an exclusive scan over the threads, the crossing bucket
  constexpr int BPT = SD_B / NT;
  const int b0 = (int)threadIdx.x * BPT;
  uint64_t mine = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) mine += h[b0 + q];
  uint64_t incl = mine;
  incl += dpp_mov64<DPP_ROW_SHR + 1>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 2>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 4>(incl);
  incl += dpp_mov64<DPP_ROW_SHR + 8>(incl);
  incl += dpp_mov64<DPP_ROW_BCAST15, 0xa>(incl);
  incl += dpp_mov64<DPP_ROW_BCAST31, 0xc>(incl);
  if (lane_id() == 63) s.red_q[wave_id()] = incl;
  __syncthreads();
  uint64_t off = 0, total = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint64_t tw = s.red_q[w];
    off += w < wave_id() ? tw : 0ull;
    total += tw;
  }
  const double tgt = target < 0 ? (double)total * (-target) : target;
  if (!(tgt > 0.0)) return radix_select<DT>(s, R, X, zlo, wmode, target, out_key);  // uniform
  const uint64_t excl = off + incl - mine;
  if ((double)excl < tgt && (double)(excl + mine) >= tgt) {  // at most one thread
    uint64_t cum = excl;
    int b = b0;
    while (b < b0 + BPT - 1 && (double)(cum + h[b]) < tgt) cum += h[b++];
    s.bc_i[0] = b;
    s.bc_q[0] = cum;
  }
  __syncthreads();
  const int bb = s.bc_i[0];
  uint64_t above = s.bc_q[0];
  if (bb < 0) return false;  // the cumulative never reaches the target (uniform)
  // the crossing bucket's keys into LDS
  auto put = [&](float x) __attribute__((always_inline)) {
    const float z = canon(x, r);
    if (z > -INFINITY && z >= zlo && dist_bucket(z, m) == bb) {
      const int i = atomicAdd(&s.bc_i[1], 1);
      if (i < SD_CAP) keys[i] = f2key(z);
    }
  };
  FOR_MEM_ELEMS(R, s, { put(x); })
  FOR_EXTRAS(s, X.n_ext, { put(x); })
  __syncthreads();
  const int n = s.bc_i[1];
  if (n > SD_CAP) return radix_select<DT>(s, R, X, zlo, wmode, target, out_key);  // uniform
  // byte radix over the staged keys; a thread merges its equal buckets before the atomic
  uint32_t prefix = 0;
#pragma unroll 1
  for (int shift = 24; shift >= 0; shift -= 8) {
    __syncthreads();
    if (threadIdx.x < 256) s.hist[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t hi_mask = (shift == 24) ? 0u : (0xffffffffu << (shift + 8));
    uint32_t cb = 0xffffffffu;
    uint64_t cw = 0;
    for (int i = threadIdx.x; i < n; i += NT) {
      const uint32_t kz = keys[i];
      if ((kz & hi_mask) == (prefix & hi_mask)) {
        const uint32_t b = (kz >> shift) & 255u;
        if (b != cb) {
          if (cw) atomicAdd((unsigned long long*)&s.hist[cb], (unsigned long long)cw);
          cb = b;
          cw = 0;
        }
        cw += weight(key2f(kz));
      }
    }
    if (cw) atomicAdd((unsigned long long*)&s.hist[cb], (unsigned long long)cw);
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t cum = above;
      int d = 255;
      for (; d >= 0; --d) {
        if ((double)(cum + s.hist[d]) >= tgt) break;
        cum += s.hist[d];
      }
      s.bc_i[0] = d;
      s.bc_q[0] = cum;
    }
    __syncthreads();
    const int d = s.bc_i[0];
    above = s.bc_q[0];
    if (d < 0) return false;  // not reached: the bucket holds the crossing
    prefix |= (uint32_t)d << shift;
  }
  __syncthreads();
  out_key = prefix;
  return true;
}

// ----------------------------------------------------------------------------------------------
// Workgroup resolution of a candidate list of at most 2 * 64 entries, by counting instead of
// sorting.  Every wave holds entries l and l + 64 in lane l and accumulates, over every NW-th list
// entry, how many entries lie strictly above each of its own (larger z) and their mass; the totals
// meet in LDS.  Then, with K, p, u of the row:
//   S2 (top-k, ties kept)  = entries with fewer than K entries strictly above, z >= the min-p bound;
//   kept (top-p)           = S2 entries whose mass strictly above is below p Z2 (so whole tie groups
//                            enter in descending z until the cumulative mass reaches p Z2; the top
//                            group always enters);
//   drawn                  = the kept entry whose id-ordered exclusive prefix of kept mass is at or
//                            below u times the kept mass, with its own mass ending above it.
// Masses are fixed point (2^24 per unit, round to nearest; every weight exp(z - m) <= 1), so every
// sum is exact and independent of the order in which the gather left the entries.
// ----------------------------------------------------------------------------------------------
constexpr int SMALL_LIST = 128;
constexpr float WFIX = 16777216.0f;        // 2^24
constexpr double WFIX40 = 1099511627776.0;  // 2^40 (kept mass reported as a float)
__device__ __forceinline__ uint32_t wfix(float w) { return (uint32_t)__builtin_fmaf(w, WFIX, 0.5f); }

// LDS totals of the counting resolver, in the general path's histogram (unused by this path)
struct CountArrays {
  uint32_t* above;  // entries strictly above (larger z)
  uint32_t* mass;   // their mass
  uint32_t* lower;  // entries at lower ids (the rank in ascending id)
  uint32_t* ties;   // entries of equal z at lower ids (top-n ranks)
};
__device__ __forceinline__ CountArrays count_arrays(Smem& s) {
  uint32_t* b = reinterpret_cast<uint32_t*>(s.hist);
  return {b, b + SMALL_LIST, b + 2 * SMALL_LIST, b + 3 * SMALL_LIST};
}
static_assert(sizeof(Smem::hist) >= 4 * SMALL_LIST * sizeof(uint32_t), "counting totals do not fit");
__device__ __forceinline__ void clear_count_arrays(Smem& s) {  // any thread set covering 0..127
  if (threadIdx.x < SMALL_LIST) reinterpret_cast<uint4*>(s.hist)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
}

// one lane's entries: z, position, fixed-point weight, presence
struct Entries {
  float z[2];
  int pos[2];
  uint32_t wf[2];
  float w[2];
  bool in[2];
};

// Accumulate over list entries i = first, first + NW, ... < n (NQ halves in use; TIE: also count
// equal z at lower ids).  Entry i is read from lane i % 64 of this wave's own registers (every wave
// holds the whole list).
template <int NQ, bool TIE>
__device__ __forceinline__ void count_above(int n, const Entries& E, uint32_t (&c)[2], uint32_t (&g)[2],
                                            uint32_t (&lo)[2], uint32_t (&t)[2]) {
  for (int i = wave_id(); i < n; i += NW) {
    const int h = i >> 6, ln = i & 63;
    const float zi = h ? lane_f32(E.z[1], ln) : lane_f32(E.z[0], ln);
    const uint32_t wi = h ? lane_u32(E.wf[1], ln) : lane_u32(E.wf[0], ln);
    const int pi = h ? lane_i32(E.pos[1], ln) : lane_i32(E.pos[0], ln);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const bool gt = zi > E.z[q];
      c[q] += gt ? 1u : 0u;
      g[q] += gt ? wi : 0u;
      lo[q] += pi < E.pos[q] ? 1u : 0u;
      if constexpr (TIE) t[q] += (zi == E.z[q] && pi < E.pos[q]) ? 1u : 0u;
    }
  }
}

// index of the first set bit over two 64-bit halves (-1 when none)
__device__ __forceinline__ int first_of2(uint64_t b0, uint64_t b1) {
  return b0 ? __ffsll((unsigned long long)b0) - 1 : (b1 ? 64 + __ffsll((unsigned long long)b1) - 1 : -1);
}

// Every thread of the workgroup calls this (it holds a barrier).  The counting is spread over all
// waves; wave 0 then decides the kept set and draws in ascending id: it scatters the kept masses to
// their id ranks and takes an exact (integer) prefix scan.  In mode 0, wave 0 receives res.id /
// res.zid; in mode 1 every thread receives the kept set's tau, zs, zmin, size (and the greedy id).
__device__ __forceinline__ Resolution resolve_count(const OutArgs& a, Smem& s, const RowState& R, const RowCtx& X,
                                                    Resolution res) {
  const int l = lane_id();
  const int n = X.n_list;
  const bool two = n > 64;
  const float m = X.m;
  const CountArrays A = count_arrays(s);
  Entries E;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int e = l + 64 * q;
    E.in[q] = e < n;
    const uint64_t k = E.in[q] ? s.sk[e] : 0ull;
    E.z[q] = E.in[q] ? cand_z(k) : -INFINITY;
    E.pos[q] = E.in[q] ? cand_pos(k) : INT32_MAX;
    E.w[q] = E.in[q] ? __expf(E.z[q] - m) : 0.f;
    E.wf[q] = E.in[q] ? wfix(E.w[q]) : 0u;
  }
  const bool rank_top = a.mode == 0 && a.n_top > 0;
  {
    uint32_t c[2] = {0u, 0u}, g[2] = {0u, 0u}, lo[2] = {0u, 0u}, t[2] = {0u, 0u};
    if (two) {
      if (rank_top) count_above<2, true>(n, E, c, g, lo, t);
      else count_above<2, false>(n, E, c, g, lo, t);
    } else {
      if (rank_top) count_above<1, true>(n, E, c, g, lo, t);
      else count_above<1, false>(n, E, c, g, lo, t);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = l + 64 * q;
      if (E.in[q]) {
        if (c[q]) atomicAdd(&A.above[e], c[q]);
        if (g[q]) atomicAdd(&A.mass[e], g[q]);
        if (lo[q]) atomicAdd(&A.lower[e], lo[q]);
        if (t[q]) atomicAdd(&A.ties[e], t[q]);
      }
    }
  }
  __syncthreads();
  if (wave_id() == 0) {
    uint32_t C[2], G[2], Q[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      C[q] = E.in[q] ? A.above[l + 64 * q] : 0xffffffffu;
      G[q] = E.in[q] ? A.mass[l + 64 * q] : 0xffffffffu;
      Q[q] = E.in[q] ? A.lower[l + 64 * q] : 0u;
    }
    bool kept[2];
    if (R.greedy) {  // the argmax with the lowest id
      const int pmin = wave_min_i(min(C[0] == 0u ? E.pos[0] : INT32_MAX, C[1] == 0u ? E.pos[1] : INT32_MAX));
#pragma unroll
      for (int q = 0; q < 2; ++q) kept[q] = E.in[q] && C[q] == 0u && E.pos[q] == pmin;
    } else {
      bool s2[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) s2[q] = E.in[q] && (!R.k_on || C[q] < (uint32_t)R.k) && E.z[q] >= X.tau_m;
      kept[0] = s2[0];
      kept[1] = s2[1];
      if (R.topp_on) {
        // G < p Z2 for an integer G is G < ceil(p Z2)
        const double Z2 = (R.k_on || R.minp_on)
                              ? (double)(uint32_t)wave_sum_i((int)((s2[0] ? E.wf[0] : 0u) + (s2[1] ? E.wf[1] : 0u)))
                              : (double)X.zfull * (double)WFIX;
        const double tg = ceil((double)R.p * Z2);
        const uint32_t target = tg <= 0.0 ? 0u : (tg >= 4294967295.0 ? 0xffffffffu : (uint32_t)tg);
#pragma unroll
        for (int q = 0; q < 2; ++q) kept[q] = s2[q] && (G[q] == 0u || G[q] < target);
      }
    }
    const uint64_t kb0 = __ballot(kept[0]), kb1 = __ballot(kept[1]);
    if (rank_top) {  // the n_top largest (ties -> lower id); padding past the list
#pragma unroll
      for (int q = 0; q < 2; ++q)
        if (E.in[q]) {
          const uint32_t r = C[q] + A.ties[l + 64 * q];
          if (r < (uint32_t)a.n_top) {
            const int64_t o = R.row * a.n_top + r;
            a.out_top_ids[o] = E.pos[q];
            a.out_top_logprobs[o] = (float)((double)E.z[q] - (double)m - X.L);
          }
        }
      if (l >= n && l < a.n_top) {
        const int64_t o = R.row * a.n_top + l;
        a.out_top_ids[o] = -1;
        a.out_top_logprobs[o] = -INFINITY;
      }
    }
    if (R.greedy) {
      const int sel = kb0 ? __ffsll((unsigned long long)kb0) - 1 : 64 + __ffsll((unsigned long long)kb1) - 1;
      res.id = sel < 64 ? lane_i32(E.pos[0], sel) : lane_i32(E.pos[1], sel - 64);
      res.zid = sel < 64 ? lane_f32(E.z[0], sel) : lane_f32(E.z[1], sel - 64);
    } else if (a.mode == 0) {
      // the draw, in ascending id over the kept entries: every entry goes to its id rank (ranks are
      // distinct: positions are), carrying its kept mass, and the cumulative of the kept masses in
      // that order is an integer prefix scan; the drawn entry is the one whose cumulative first
      // exceeds u times the kept mass
      uint32_t* dw = A.mass;  // reused: wave 0 alone reads and writes it from here on
      int32_t* dp = reinterpret_cast<int32_t*>(A.ties);
#pragma unroll
      for (int q = 0; q < 2; ++q)
        if (E.in[q]) {
          dw[Q[q]] = kept[q] ? E.wf[q] : 0u;
          dp[Q[q]] = l + 64 * q;  // the entry, by its lane and half
        }
      uint32_t wk[2], cu[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) wk[q] = l + 64 * q < n ? dw[l + 64 * q] : 0u;
      cu[0] = wave_incl_scan_u(wk[0]);
      cu[1] = lane_u32(cu[0], 63) + wave_incl_scan_u(wk[1]);
      const uint32_t total = two ? lane_u32(cu[1], 63) : lane_u32(cu[0], 63);
      uint32_t tf = (uint32_t)((double)R.u * (double)total);
      if (tf >= total) tf = total - 1u;
      const int r = first_of2(__ballot(cu[0] > tf), __ballot(l + 64 < n && cu[1] > tf));
      if (r >= 0) {
        const int e = dp[r];
        res.id = e < 64 ? lane_i32(E.pos[0], e) : lane_i32(E.pos[1], e - 64);
        res.zid = e < 64 ? lane_f32(E.z[0], e) : lane_f32(E.z[1], e - 64);
      }
    }
    if (a.mode == 1) {
      res.kept = __popcll(kb0) + __popcll(kb1);
      res.zmin = wave_min(fminf(kept[0] ? E.z[0] : INFINITY, kept[1] ? E.z[1] : INFINITY));
      uint64_t w40 = 0;
#pragma unroll
      for (int q = 0; q < 2; ++q)
        if (kept[q]) w40 += (uint64_t)__builtin_fma((double)E.w[q], WFIX40, 0.5);
      res.zs = (float)((double)wave_sum_u64(w40) / WFIX40);
      if (l == 0) {
        s.bc_f[0] = res.zmin;
        s.bc_f[1] = res.zs;
        s.bc_i[1] = res.kept;
        s.bc_i[0] = res.id;
      }
    }
  }
  if (a.mode == 1) {  // every thread needs the kept set for the dense output
    __syncthreads();
    res.zmin = s.bc_f[0];
    res.zs = s.bc_f[1];
    res.kept = s.bc_i[1];
    res.id = s.bc_i[0];
  }
  res.tau = res.zmin;
  res.id_here = 1;
  return res;
}

// ----------------------------------------------------------------------------------------------
// List path: exact resolution on the sorted candidate list (leader workgroup only)
// ----------------------------------------------------------------------------------------------
__device__ __noinline__ Resolution resolve_list(const OutArgs a, Smem& s, const RowState R, const RowCtx X,
                                          Resolution res) {
  const int n = X.n_list;
  const float m = X.m;
  const int npad = next_pow2(n);
  for (int i = n + threadIdx.x; i < npad; i += NT) s.sk[i] = 0;  // key 0 sorts last
  bitonic_sort(s, npad, true);  // descending z, then ascending position
  for (int i = threadIdx.x; i < n; i += NT) {
    const float z = cand_z(s.sk[i]);
    s.l_z[i] = z;
    s.l_p[i] = cand_pos(s.sk[i]);
    s.l_w[i] = __expf(z - m);
  }
  __syncthreads();
  // thread t owns entries [EPT t, EPT t + EPT) in every scan below (fixed structure); an entry's
  // cumulative is the thread's exclusive prefix plus the serial sum of its own entries
  const int i0 = EPT * (int)threadIdx.x;
  float cm[EPT];
  int nS;
  if (R.greedy) {
    nS = 1;
  } else {
    float tau2 = X.tau_m;
    if (R.k_on && R.k <= n) tau2 = fmaxf(tau2, s.l_z[R.k - 1]);
    int loc = 0;
#pragma unroll
    for (int q = 0; q < EPT; ++q) loc += (i0 + q < n && s.l_z[i0 + q] >= tau2) ? 1 : 0;
    const int n2 = block_sum_i(loc, s);  // S2 is a prefix of the descending list
    nS = n2;
    if (R.topp_on) {
      float ts = 0.f;
#pragma unroll
      for (int q = 0; q < EPT; ++q) ts += (i0 + q < n2) ? s.l_w[i0 + q] : 0.f;
      float tot;
      float cum = block_excl_scan(ts, s, &tot);
#pragma unroll
      for (int q = 0; q < EPT; ++q) {
        cum += (i0 + q < n2) ? s.l_w[i0 + q] : 0.f;
        cm[q] = cum;
        if (i0 + q == n2 - 1) s.bc_f[0] = cum;  // Z2: cumulative at the last S2 entry
      }
      __syncthreads();
      const float Z2 = (R.k_on || R.minp_on) ? s.bc_f[0] : X.zfull;
      const float target = R.p * Z2;
      int first = INT32_MAX;
#pragma unroll
      for (int q = 0; q < EPT; ++q)
        if (first == INT32_MAX && i0 + q < n2 && cm[q] >= target) first = i0 + q;
      first = block_min_i(first, s);
      if (first != INT32_MAX) {  // the nucleus closes at the end of that tie group
        const float zc = s.l_z[first];
        int cnt = 0;
#pragma unroll
        for (int q = 0; q < EPT; ++q) cnt += (i0 + q < n2 && s.l_z[i0 + q] >= zc) ? 1 : 0;
        nS = block_sum_i(cnt, s);
      }
    }
  }
  res.kept = nS;
  res.zmin = s.l_z[nS - 1];
  res.tau = res.zmin;
  {
    float ts = 0.f;
#pragma unroll
    for (int q = 0; q < EPT; ++q) ts += (i0 + q < nS) ? s.l_w[i0 + q] : 0.f;
    float tot;
    float cum = block_excl_scan(ts, s, &tot);
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      cum += (i0 + q < nS) ? s.l_w[i0 + q] : 0.f;
      if (i0 + q == nS - 1) s.bc_f[1] = cum;
    }
    __syncthreads();
    res.zs = s.bc_f[1];
  }
  res.id_here = 1;
  if (R.greedy) {
    res.id = s.l_p[0];
    res.zid = s.l_z[0];
  } else if (a.mode == 0) {
    // inverse CDF in ascending token id over the kept prefix: sort (position, index) pairs
    const int npS = next_pow2(nS);
    __syncthreads();
    for (int i = threadIdx.x; i < npS; i += NT)
      s.sk[i] = i < nS ? (((uint64_t)(uint32_t)s.l_p[i] << 32) | (uint32_t)i) : ~0ull;
    bitonic_sort(s, npS, false);
    float wv[EPT];
    float ts = 0.f;
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      wv[q] = (i0 + q < nS) ? s.l_w[(uint32_t)s.sk[i0 + q]] : 0.f;
      ts += wv[q];
    }
    float tot;
    float cum = block_excl_scan(ts, s, &tot);
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
      cum += wv[q];
      cm[q] = cum;
      if (i0 + q == nS - 1) s.bc_f[2] = cum;  // the id-order total
    }
    __syncthreads();
    const float t = R.u * s.bc_f[2];
    int first = INT32_MAX;
#pragma unroll
    for (int q = 0; q < EPT; ++q)
      if (first == INT32_MAX && i0 + q < nS && cm[q] > t) first = i0 + q;
    first = block_min_i(first, s);
    if (first == INT32_MAX) {  // rounding left the cumulative at u: the last positive weight
      int last = -1;
#pragma unroll
      for (int q = 0; q < EPT; ++q)
        if (i0 + q < nS && wv[q] > 0.f) last = i0 + q;
      first = block_max_i(last, s);
    }
    if (first >= 0) {
      const int di = (int)(uint32_t)s.sk[first];
      res.id = s.l_p[di];
      res.zid = s.l_z[di];
    }
  }
  // top-n straight from the descending list
  if (a.mode == 0 && a.n_top > 0) {
    for (int t = threadIdx.x; t < a.n_top; t += NT) {
      const int64_t o = R.row * a.n_top + t;
      if (t < n) {
        a.out_top_ids[o] = s.l_p[t];
        a.out_top_logprobs[o] = (float)((double)s.l_z[t] - (double)m - X.L);
      } else {
        a.out_top_ids[o] = -1;
        a.out_top_logprobs[o] = -INFINITY;
      }
    }
  }
  __syncthreads();
  return res;
}

// ----------------------------------------------------------------------------------------------
// General path (every chunk of the row): thresholds by radix selection, draw through an id-ordered
// weight buffer in the workspace, top-n by a separate candidate list (selection for massive ties)
// ----------------------------------------------------------------------------------------------
template <class DT>
__device__ __noinline__ Resolution resolve_general(const OutArgs a, Smem& s, const RowState R, const RowCtx X,
                                             Resolution res) {
  const float r = R.r, m = X.m;
  const int P = R.P, c = R.c;
  const bool leader = c == 0;
  const int n_ext = X.n_ext;
  float tau_star;
  if (R.greedy) {
    tau_star = m;
  } else {
    float tau2 = X.tau_m;
    uint32_t kk = 0;
    auto select = [&](float zlo, int wmode, double target, uint32_t& key) -> bool {
      return P == 1 ? select_dist<DT>(s, R, X, zlo, wmode, target, key)
                    : radix_select<DT>(s, R, X, zlo, wmode, target, key);
    };
    if (R.k_on && select(-INFINITY, 0, (double)R.k, kk)) tau2 = fmaxf(tau2, key2f(kk));
    tau_star = tau2;
    if (R.topp_on && select(tau2, 1, -(double)R.p, kk)) tau_star = fmaxf(tau_star, key2f(kk));
  }
  // kept count, min z and fixed-point mass of S = {finite z >= tau_star}; greedy argmax position.  A
  // sampled (mode 0) row that is not greedy reports none of them, so it skips this pass.
  int kept = 0, best = INT32_MAX;
  float zmin = INFINITY;
  uint64_t zsx = 0;
  if (a.mode == 1 || R.greedy) {  // uniform over the workgroup
  FOR_MEM_ELEMS(R, s, {
    const float z = canon(x, r);
    if (z > -INFINITY && z >= tau_star) {
      ++kept;
      zmin = fminf(zmin, z);
      zsx += fixmass(__expf(z - m));
      if (z == m && pos < best) best = pos;
    }
  })
  FOR_EXTRAS(s, n_ext, {
    const float z = canon(x, r);
    if (z > -INFINITY && z >= tau_star) {
      ++kept;
      zmin = fminf(zmin, z);
      zsx += fixmass(__expf(z - m));
      if (z == m && pos < best) best = pos;
    }
  })
  kept = block_sum_i(kept, s);
  zmin = block_min(zmin, s);
  zsx = block_sum_u64(zsx, s);
  best = block_min_i(best, s);
  }
  // draw: blocked scans in ascending id over this chunk's region [lo, hi), reading the logits back
  const int64_t lo = R.owns_head ? 0 : (int64_t)R.head + R.s0 * DT::VEC;
  const int64_t hi = R.owns_tail ? (int64_t)R.V : (int64_t)R.head + R.s1 * DT::VEC;
  const bool draw = (a.mode == 0) && !R.greedy;
  // The region in groups of GS consecutive positions (GS = 16, doubled until the group weights fit
  // the slot-code area, which is free once the candidates are gathered): every group's weight summed
  // in position order, the group weights summed in order per thread over a contiguous run of groups,
  // an exclusive scan over the threads, then the crossing thread walks its run and the crossing group.
  // An element's cumulative is thus (thread prefix + earlier groups of its run + earlier elements of
  // its group), the same expression for the search and for the totals.  Each element is loaded
  // unconditionally (its extras value replaces it where it has one), so a group's loads are in
  // flight together.
  float ctot = 0.f;
  int clast = -1;
  float* gw = reinterpret_cast<float*>(s.scode);
  constexpr int GMAX = (int)(sizeof(s.scode) / sizeof(float));
  int gsz = 16;
  while ((hi - lo + gsz - 1) / gsz > GMAX) gsz *= 2;
  const int ng = (int)((hi - lo + gsz - 1) / gsz);
  auto elem_w = [&](int64_t i) __attribute__((always_inline)) -> float {
    const int pos = (int)(i < hi ? i : lo);
    const int u = n_ext > 0 ? extras_index<DT>(s, R, pos) : -1;
    const float raw = load_pos<DT>(R, pos);
    const float z = canon(u >= 0 ? s.x_val[u] : raw, r);
    return (i < hi && z > -INFINITY && z >= tau_star) ? __expf(z - m) : 0.f;
  };
  auto group_w = [&](int g, int* lp) __attribute__((always_inline)) -> float {
    const int64_t p0 = lo + (int64_t)g * gsz;
    float w = 0.f;
    for (int q0 = 0; q0 < gsz; q0 += 16) {
      float wq[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) wq[q] = elem_w(p0 + q0 + q);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        w += wq[q];
        if (wq[q] > 0.f) *lp = (int)(p0 + q0 + q);
      }
    }
    return w;
  };
  bool weights_done = false;
  auto scan_find = [&](float target) -> int {
    if (!weights_done) {
      int lp = -1;
      for (int g = threadIdx.x; g < ng; g += NT) gw[g] = group_w(g, &lp);
      clast = block_max_i(lp, s);  // its barriers also publish gw
      weights_done = true;
    }
    const int per = (ng + NT - 1) / NT;
    const int g0 = (int)threadIdx.x * per, g1 = min(g0 + per, ng);
    float mine = 0.f;
    for (int g = g0; g < g1; ++g) mine += gw[g];
    float btot;
    float cum = block_excl_scan(mine, s, &btot);
    ctot = btot;
    int f = INT32_MAX;
    if (cum + mine > target) {
      int g = g0;
      while (g < g1 - 1 && cum + gw[g] <= target) cum += gw[g++];
      const int64_t p0 = lo + (int64_t)g * gsz;
      for (int q = 0; q < gsz && p0 + q < hi; ++q) {
        const float w = elem_w(p0 + q);
        cum += w;
        if (w > 0.f && cum > target) {  // a later thread that starts above the target takes its
          f = (int)(p0 + q);            // first kept element: the minimum over threads decides
          break;
        }
      }
    }
    f = block_min_i(f, s);
    return f == INT32_MAX ? -1 : f;
  };
  if (draw) (void)scan_find(INFINITY);
  // per-chunk results, combined in chunk order (identical arithmetic in every chunk)
  float cum_before = 0.f, row_tot = ctot;
  int kept_row = kept, last_row = clast, best_row = best, c_star = -1;
  float zmin_row = zmin;
  uint64_t zsx_row = zsx;
  if (P > 1) {
    if (threadIdx.x == 0) {
      st_agent(&X.gstats[c].w_total, ctot);
      st_agent(&X.gstats[c].last_pos, (int32_t)clast);
      st_agent(&X.gstats[c].n_keep, (int32_t)kept);
      st_agent(&X.gstats[c].zmin, zmin);
      st_agent(&X.gstats[c].zs_fix, zsx);
      st_agent(&X.gstats[c].best, (int32_t)best);
    }
    group_barrier(X.gsync, P);
    float cum = 0.f;
    float cums[MAXP];
    kept_row = 0;
    zmin_row = INFINITY;
    last_row = -1;
    best_row = INT32_MAX;
    zsx_row = 0;
    for (int q = 0; q < P; ++q) {
      cum = cum + ld_agent(&X.gstats[q].w_total);
      cums[q] = cum;
      kept_row += ld_agent(&X.gstats[q].n_keep);
      zmin_row = fminf(zmin_row, ld_agent(&X.gstats[q].zmin));
      last_row = max(last_row, (int)ld_agent(&X.gstats[q].last_pos));
      best_row = min(best_row, (int)ld_agent(&X.gstats[q].best));
      zsx_row += ld_agent(&X.gstats[q].zs_fix);
    }
    row_tot = cum;
    const float tt = R.u * row_tot;
    for (int q = 0; q < P; ++q)
      if (c_star < 0 && cums[q] > tt) c_star = q;
    cum_before = c > 0 ? cums[c - 1] : 0.f;
    group_barrier(X.gsync, P);  // stats read before the top-n stage reuses them
  } else {
    c_star = (ctot > R.u * ctot) ? 0 : -1;
  }
  res.tau = tau_star;
  res.kept = kept_row;
  res.zmin = zmin_row;
  res.zs = (float)((double)zsx_row / FIX_SCALE);
  res.id_here = 0;
  if (R.greedy) {
    res.id = best_row;
    res.zid = m;
    res.kept = 1;
    res.zmin = m;
    res.tau = m;
    res.zs = 1.0f;
    res.id_here = leader;
  } else if (draw) {
    const float tt = R.u * row_tot;
    int idf = -1;
    if (c == c_star) {
      idf = scan_find(tt - cum_before);
      if (idf < 0) idf = clast;  // rounding inside the chunk: its last positive weight
    } else if (c_star < 0 && clast >= 0 && clast == last_row) {
      idf = clast;  // rounding beyond the row total: the row's last positive weight
    }
    if (idf >= 0) {
      res.id = idf;
      res.zid = canon(x_at<DT>(s, R, n_ext, idf), r);
      res.id_here = 1;
    }
  }
  // top-n: the n_top largest (z desc, position asc)
  if (a.mode == 0 && a.n_top > 0) {
    const int nt = a.n_top;
    const float bl = X.row_beta;
    bool tover = !(bl > -INFINITY);
    int nl = tover ? 0 : gather_mem<DT>(s, R, n_ext, bl, false);
    tover = tover || nl > LCAP;
    if (P > 1) nl = union_lists(s, R, X, nl, tover);
    if (tover) {
      // selection: tau_n = n-th largest z, the entries strictly above it, then ties by position
      uint32_t kk = 0;
      const bool ok = radix_select<DT>(s, R, X, -INFINITY, 0, (double)nt, kk);
      const float tau_n = ok ? key2f(kk) : -INFINITY;
      int ngt = gather_mem<DT>(s, R, n_ext, tau_n, true);  // fewer than nt entries
      if (P > 1) {
        bool of2 = false;
        ngt = union_lists(s, R, X, ngt, of2);
      }
      int last = -1;
      for (int q = ngt; q < nt; ++q) {
        int bp = INT32_MAX;
        if (tau_n > -INFINITY) {
          FOR_MEM_ELEMS(R, s, {
            if (canon(x, r) == tau_n && pos > last && pos < bp) bp = pos;
          })
          FOR_EXTRAS(s, n_ext, {
            if (canon(x, r) == tau_n && pos > last && pos < bp) bp = pos;
          })
        }
        bp = block_min_i(bp, s);
        if (P > 1) {
          if (threadIdx.x == 0) st_agent(&X.gstats[c].last_pos, (int32_t)bp);
          group_barrier(X.gsync, P);
          int b2 = INT32_MAX;
          for (int qq = 0; qq < P; ++qq) b2 = min(b2, (int)ld_agent(&X.gstats[qq].last_pos));
          bp = b2;
          group_barrier(X.gsync, P);
        }
        if (bp == INT32_MAX) break;
        if (leader && threadIdx.x == 0) s.sk[q] = cand_key(tau_n, bp);
        __syncthreads();
        last = bp;
        ngt = q + 1;
      }
      nl = ngt;
    }
    if (leader) write_top_n(a, s, X, R.row, min(nl, LCAP));
  }
  __syncthreads();
  return res;
}

// ----------------------------------------------------------------------------------------------
// Dense filtered distribution (albireo_topk_topp), written by every chunk from memory
// ----------------------------------------------------------------------------------------------
template <class DT>
__device__ __noinline__ void dense_probs(const OutArgs a, Smem& s, const RowState R, const RowCtx X,
                                         Resolution res, bool skip, bool broadcast) {
  if (broadcast) {  // list path with P > 1: the leader resolved alone
    if (R.c == 0 && threadIdx.x == 0) {
      st_agent(&X.gres->tau, res.tau);
      st_agent(&X.gres->zs, res.zs);
      st_agent(&X.gres->id, (int32_t)res.id);
    }
    group_barrier(X.gsync, R.P);
    res.tau = ld_agent(&X.gres->tau);
    res.zs = ld_agent(&X.gres->zs);
    res.id = ld_agent(&X.gres->id);
    group_barrier(X.gsync, R.P);
  }
  float* orow = a.out_probs + R.row * a.V;
  const float r = R.r, m = X.m;
  const float inv = (skip || !(res.zs > 0.f)) ? 0.f : 1.0f / res.zs;
  const float tau = res.tau;
  const int id = res.id;
  const bool greedy = R.greedy;
  FOR_MEM_ELEMS(R, s, {
    const float z = canon(x, r);
    float pr = 0.f;
    if (!skip) {
      if (greedy) pr = (pos == id) ? 1.0f : 0.f;
      else if (z > -INFINITY && z >= tau) pr = __expf(z - m) * inv;
    }
    orow[pos] = pr;
  })
  __threadfence_block();
  __syncthreads();
  FOR_EXTRAS(s, X.n_ext, {  // penalised body entries overwrite; head/tail entries are written here
    const float z = canon(x, r);
    float pr = 0.f;
    if (!skip) {
      if (greedy) pr = (pos == id) ? 1.0f : 0.f;
      else if (z > -INFINITY && z >= tau) pr = __expf(z - m) * inv;
    }
    orow[pos] = pr;
  })
  __syncthreads();
}

// Wait (bounded) until the row's penalty state has reached the given level of the LDS counter: one
// count per wave that has marked its share of the history, then one for wave 0's finished presence
// bitmap, then one for its extras numbering and cleared counts.
// A wait that gives up sets FLAG_TIMEOUT in the row's LDS flags.
__device__ __forceinline__ void wait_ready(Smem& s, uint32_t level) {
  for (uint32_t n = 0; n < SPIN_LIMIT; ++n) {
    if (__hip_atomic_load(&s.ready, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= level) return;
    __builtin_amdgcn_s_sleep(1);
  }
  atomicOr(&s.flags, FLAG_TIMEOUT);
}

// Whether a history id lies in this chunk (the chunk's body slots, or the head / tail it owns).
template <class DT>
__device__ __forceinline__ bool id_in_chunk(const RowState& R, int id) {
  if (id < R.head) return R.owns_head;
  if (id >= R.tail_lo) return R.owns_tail;
  const int64_t slot = (id - R.head) / DT::VEC;
  return slot >= R.s0 && slot < R.s1;
}

// Add one history occurrence to its extras entry: ids outside [0, V) (flagged by the presence build),
// ids of other chunks and ids cut for capacity have none.
template <class DT>
__device__ __forceinline__ void count_history_id(Smem& s, const RowState& R, int id) {
  if ((unsigned)id >= (unsigned)R.V) return;
  const int u = extras_index<DT>(s, R, id);
  if (u < 0) return;
  atomicAdd(&s.x_cnt[u], 1u);
  s.x_pos[u] = id;  // every counting thread of this id writes the same value
}

// s_waitcnt immediate for vmcnt(0) alone (expcnt and lgkmcnt at their maxima)
constexpr int WAIT_VM0 = 0x0F70;
constexpr int HSTAGE = 3 * LCAP;  // history ids staged in LDS at once (the list arrays, unused until
                                  // the candidate list is resolved)

__device__ __forceinline__ int32_t* hist_stage(Smem& s) { return reinterpret_cast<int32_t*>(s.l_z); }
static_assert(offsetof(Smem, l_w) == offsetof(Smem, l_z) + LCAP * 4 &&
                  offsetof(Smem, l_p) == offsetof(Smem, l_w) + LCAP * 4,
              "the history staging area spans l_z, l_w and l_p");

// Stage history ids [b, b + n) (n <= HSTAGE) in LDS with direct-to-LDS loads: no registers are
// involved, so nothing can be re-issued or moved behind the row loads.
__device__ __forceinline__ void stage_history(Smem& s, const int32_t* hist_ids, int64_t b, int n) {
  const uint64_t hb = reinterpret_cast<uint64_t>(hist_ids + b);
  const uint32_t hb_lo = __builtin_amdgcn_readfirstlane((uint32_t)hb);
  const uint32_t hb_hi = __builtin_amdgcn_readfirstlane((uint32_t)(hb >> 32));
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      reinterpret_cast<void*>(((uint64_t)hb_hi << 32) | hb_lo), (short)0, __builtin_amdgcn_readfirstlane(n * 4),
      0x00020000);
  int32_t* hst = hist_stage(s);
  const int lane = lane_id();
  const int nk = __builtin_amdgcn_readfirstlane((n + 63) / 64);
  for (int k = 0; k < nk; ++k)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(hst + 64 * k), 4,
                                             (lane + 64 * k) * 4, 0, 0, 0);
}

// Chunk-relative position of a row id's register element: (slot << 3) | element, or -1 when the id
// is not a body element of this chunk.  32-bit arithmetic throughout (V < 2^31).
template <class DT>
__device__ __forceinline__ int body_code(const RowState& R, int id) {
  const int rel = id - R.head;
  if (rel < 0 || id >= R.tail_lo) return -1;
  const int sl = rel / DT::VEC - (int)R.s0;  // rel >= 0: a shift
  if ((unsigned)sl >= (unsigned)(R.s1 - R.s0)) return -1;
  return (sl << 3) | (rel % DT::VEC);
}

// Wave 0, once every wave has marked its share of the history in the presence bitmap: mark the rest
// of a history longer than the staging area, apply the capacity cut, and advance the flag (to 9), which
// lets the other waves mask their registers.  When the history could name more distinct ids than the
// extras hold, only the lowest positions keep their bit (the rest keep their raw value: penalties not
// applied, LIMIT flagged).  Returns the flags found.
template <class DT>
__device__ __forceinline__ uint32_t finish_presence(Smem& s, const RowState& R, const int32_t* hist_ids) {
  const int lane = lane_id();
  const int n_ht = (R.owns_head ? R.head : 0) + (R.owns_tail ? R.V - R.tail_lo : 0);
  uint32_t flags = 0;
  if (R.pen_on) {
    const int32_t* hst = hist_stage(s);
    for (int64_t b = R.h_lo + HSTAGE; b < R.h_hi; b += HSTAGE) {  // long histories only
      const int n = (int)min<int64_t>(R.h_hi - b, HSTAGE);
      stage_history(s, hist_ids, b, n);
      for (int i = lane; i < n; i += 64) {
        const int id = hst[i];
        if ((unsigned)id >= (unsigned)R.V) {
          flags = FLAG_BAD_INPUT;
        } else {
          const int code = body_code<DT>(R, id);
          if (code >= 0) atomicOr(&s.bitmap[code >> 5], 1u << (code & 31));
        }
      }
      // the direct-to-LDS loads are complete here, so the publication below waits for LDS only
      __builtin_amdgcn_s_waitcnt(WAIT_VM0);
    }
    flags = wave_or(flags);
    const uint32_t cap = (uint32_t)(UCAP - n_ht);
    if ((uint64_t)(R.h_hi - R.h_lo) > cap) {
      // distinct body ids = set bits; each lane owns WPL consecutive words (position order)
      constexpr int WPL = NWORDS / 64;
      uint32_t cnt = 0;
      for (int i = lane * WPL; i < (lane + 1) * WPL; ++i) cnt += __popc(s.bitmap[i]);
      const uint32_t incl = wave_incl_scan_u(cnt);
      if (lane_u32(incl, 63) > cap) {
        flags |= FLAG_LIMIT;
        uint32_t before = incl - cnt;  // keep the lowest positions within the capacity
        for (int i = lane * WPL; i < (lane + 1) * WPL; ++i) {
          uint32_t wv = s.bitmap[i];
          const uint32_t c = __popc(wv);
          if (before + c > cap) {
            uint32_t keep = before >= cap ? 0u : cap - before;
            uint32_t out = 0;
            while (keep > 0 && wv) {
              const uint32_t lowbit = wv & (0u - wv);
              out |= lowbit;
              wv ^= lowbit;
              --keep;
            }
            s.bitmap[i] = out;
          }
          before += c;
        }
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");  // LDS only: row loads stay in flight
  if (lane == 0) atomicAdd(&s.ready, 1u);
  return flags;
}


// Wave 0, second: number the extras entries (penalised body elements by position, through the word
// prefixes of the bitmap, then the unaligned head / tail positions the chunk owns), clear their
// counts and advance the flag (to 10 when penalties are on).  A history longer than the staging area is also counted here;
// otherwise every thread counts its share of the staged history after its online pass.
template <class DT>
__device__ __forceinline__ void build_ranks(Smem& s, const RowState& R, const int32_t* hist_ids, uint32_t flags) {
  const int lane = lane_id();
  const int n_head = R.owns_head ? R.head : 0;
  const int n_ht = n_head + (R.owns_tail ? R.V - R.tail_lo : 0);
  int n_body = 0;
  if (R.pen_on) {
    constexpr int WPL = NWORDS / 64;
    static_assert(WPL * 64 == NWORDS && WPL % 4 == 0, "bitmap words do not split evenly over the lanes");
    const uint4* own = reinterpret_cast<const uint4*>(s.bitmap + lane * WPL);
    uint32_t cnt = 0;
#pragma unroll 4
    for (int i = 0; i < WPL / 4; ++i) {
      const uint4 w = own[i];
      cnt += __popc(w.x) + __popc(w.y) + __popc(w.z) + __popc(w.w);
    }
    const uint32_t incl = wave_incl_scan_u(cnt);
    n_body = (int)lane_u32(incl, 63);
    uint32_t before = incl - cnt;
    uint2* pref = reinterpret_cast<uint2*>(s.wpref + lane * WPL);  // 4 prefixes per 8-byte store
#pragma unroll 4
    for (int i = 0; i < WPL / 4; ++i) {
      const uint4 w = own[i];
      const uint32_t p0 = before;
      const uint32_t p1 = p0 + __popc(w.x);
      const uint32_t p2 = p1 + __popc(w.y);
      const uint32_t p3 = p2 + __popc(w.z);
      before = p3 + __popc(w.w);
      pref[i] = make_uint2(p0 | (p1 << 16), p2 | (p3 << 16));
    }
  }
  for (int i = lane; i < n_body + n_ht; i += 64) s.x_cnt[i] = 0u;
  for (int i = lane; i < n_ht; i += 64) s.x_pos[n_body + i] = i < n_head ? i : R.tail_lo + (i - n_head);
  if (lane == 0) {
    s.n_body = n_body;
    s.n_ext = n_body + n_ht;
    if (flags) atomicOr(&s.flags, flags);
  }
  if (R.pen_on && R.h_hi - R.h_lo > HSTAGE) {  // long history: counted here, batch by batch
    const int32_t* hst = hist_stage(s);
    for (int64_t b = R.h_lo; b < R.h_hi; b += HSTAGE) {
      const int n = (int)min<int64_t>(R.h_hi - b, HSTAGE);
      stage_history(s, hist_ids, b, n);
      for (int i = lane; i < n; i += 64) count_history_id<DT>(s, R, hst[i]);
    }
    __builtin_amdgcn_s_waitcnt(WAIT_VM0);  // as in finish_presence
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");  // LDS only: row loads stay in flight
  if (lane == 0) atomicAdd(&s.ready, 1u);
}

// K-th bound from the workgroup histogram of per-thread maxima: the bucket holding the K-th largest
// (counting from the top bucket), then the smallest maximum at or above that bucket.  Every wave
// evaluates it on the same LDS data, so no further barrier is needed.
__device__ __forceinline__ float kth_from_hist(const Smem& s, int K) {
  const int l = lane_id();
  const uint32_t c0 = s.kh_cnt[255 - 4 * l], c1 = s.kh_cnt[254 - 4 * l], c2 = s.kh_cnt[253 - 4 * l],
                 c3 = s.kh_cnt[252 - 4 * l];
  const uint32_t own = c0 + c1 + c2 + c3;
  const uint32_t incl = wave_incl_scan_u(own);
  const uint64_t hit = __ballot(incl >= (uint32_t)K);
  if (!hit) return -INFINITY;
  const int first = __ffsll((unsigned long long)hit) - 1;
  int c = 0;
  {
    uint32_t cum = incl - own;
    if ((cum += c0) >= (uint32_t)K) c = 255 - 4 * l;
    else if ((cum += c1) >= (uint32_t)K) c = 254 - 4 * l;
    else if ((cum += c2) >= (uint32_t)K) c = 253 - 4 * l;
    else c = 252 - 4 * l;
  }
  c = lane_i32(c, first);
  uint32_t mk = 0xffffffffu;
  if (255 - 4 * l >= c) mk = min(mk, s.kh_min[255 - 4 * l]);
  if (254 - 4 * l >= c) mk = min(mk, s.kh_min[254 - 4 * l]);
  if (253 - 4 * l >= c) mk = min(mk, s.kh_min[253 - 4 * l]);
  if (252 - 4 * l >= c) mk = min(mk, s.kh_min[252 - 4 * l]);
  return key2f(wave_min_u32(mk));
}

// ----------------------------------------------------------------------------------------------
// The sampling kernel (mode 0) / filtered-distribution kernel (mode 1)
// ----------------------------------------------------------------------------------------------
// One row chunk end to end.  MULTI selects the build for P > 1 chunks per row (cross-workgroup
// exchanges through the workspace); the single-chunk build has none of that code.
template <class DT, int J, bool MULTI, bool SEG>
__device__ __forceinline__ void process_row(const KArgs& a, Smem& s, RowCtx& X, int64_t row, int c) {
  const int P = MULTI ? a.P : 1;
  const bool leader = (c == 0);
  {
    RowState R;
    row_geometry<DT, SEG>(a, row, c, R);
    R.P = P;

    // ---------------- row loads first ----------------
    // The row loads depend on the kernel arguments only, so they go out before anything else.  They
    // are software-pipelined with the online pass: slot j + PIPE is issued just before slot j is
    // consumed, so each wave computes on its data as it arrives, with enough bytes in flight to hold
    // the HBM stream.  Every issue is unconditional: a load under a branch would have its register
    // merged at the join, which waits for the load.
    Chunk<DT, J> ch;
    constexpr int PIPE = J < 8 ? J : 8;
    constexpr int JLO = MULTI ? 0 : live_slots_min(J);
    const int nslots = (int)(R.s1 - R.s0);
    // one buffer resource per chunk (SGPRs) and a 32-bit lane offset; its inputs are made visibly
    // wave-uniform so the descriptor lives in SGPRs
    const int64_t off_s0 = slot_off<DT>(R, R.s0);
    const uint64_t cb = reinterpret_cast<uint64_t>(R.rowp + off_s0);
    const uint32_t cb_lo = __builtin_amdgcn_readfirstlane((uint32_t)cb);
    const uint32_t cb_hi = __builtin_amdgcn_readfirstlane((uint32_t)(cb >> 32));
    // bytes from the chunk's first slot to the end of its last (the host keeps this below 2^31)
    const uint32_t span = SEG ? (nslots > 0 ? (uint32_t)(slot_off<DT>(R, R.s1 - 1) + 16 - off_s0) : 0u)
                              : (uint32_t)nslots * 16u;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(((uint64_t)cb_hi << 32) | cb_lo), (short)0,
        __builtin_amdgcn_readfirstlane(span), 0x00020000);
    const int voff = (int)threadIdx.x * 16;
    // Blocked layout: each thread tracks its slot's place in its block (sr) and the slot's byte
    // offset from the chunk base (soff), advanced by NT slots per issue; offsets grow with the slot,
    // so slots past the chunk still land past the range and read as 0.  The host checks that the
    // offsets of all J slots stay below 2^32.
    uint32_t sr = 0, soff = 0;
    const uint32_t sgap = (uint32_t)R.sgap, sps = a.seg_sps, ntr = a.seg_ntr;
    const uint32_t step0 = (uint32_t)NT * 16u + a.seg_ntq * sgap, step1 = step0 + sgap;
    if constexpr (SEG) {
      const uint32_t q0 = (uint32_t)R.s0 + threadIdx.x;
      const uint32_t g0 = seg_of(R, q0);
      sr = q0 - g0 * sps;
      soff = (uint32_t)voff + (g0 - seg_of(R, (uint32_t)R.s0)) * sgap;
    }
    // Unconditional loads with the whole offset in the range-checked VGPR operand: slots past the
    // chunk read as 0 without touching memory and are set to -inf when consumed (only the last,
    // partly filled slots can be affected).  Slots are issued in order j = 0, 1, ..., J - 1.
    auto issue = [&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      uint32_t off = (uint32_t)(voff + j * NT * 16);
      if constexpr (SEG) {
        if constexpr (j > 0) {
          sr += ntr;
          const bool w = sr >= sps;
          sr = w ? sr - sps : sr;
          soff += w ? step1 : step0;
        }
        off = soff;
      }
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0);
      ch.template set<j>(make_uint4(v[0], v[1], v[2], v[3]));
    };
    // the parameter loads (scalar) go out first, then the first row slots; the rest of the pipeline
    // is issued once the history has been sent, so that it is not queued behind the whole initial
    // burst of row loads across the chip
    constexpr int PIPE0 = PIPE < 2 ? PIPE : 2;
    const RawParams rp = row_params_load(a, row);
    static_for<PIPE0>(issue);
    row_params(a, rp, R);
    // the unaligned head / tail elements this chunk owns (the extras entries after the penalised
    // body ones), loaded now and staged after the online pass: one unconditional load per thread
    const int n_head0 = R.owns_head ? R.head : 0;
    const int n_ht0 = n_head0 + (R.owns_tail ? R.V - R.tail_lo : 0);
    const float xht = load_pos<DT>(
        R, (int)threadIdx.x < n_ht0 ? ((int)threadIdx.x < n_head0 ? (int)threadIdx.x
                                                                       : R.tail_lo + ((int)threadIdx.x - n_head0))
                                         : 0);
    const bool extras_any = R.pen_on || (R.owns_head && R.head > 0) || (R.owns_tail && R.tail_lo < R.V);
    const bool builder = extras_any && wave_id() == 0;
    const int64_t n_hist = R.h_hi - R.h_lo;

    // ---------------- penalty state ----------------
    // Every wave marks its share of the history in the presence bitmap of penalised register elements
    // (and stages it in LDS for the counts) and advances an LDS counter; at 8, wave 0 applies the
    // capacity rule and advances it to 9, which is all the waves need before their online pass, then
    // numbers the extras entries (10).  Every thread counts its share of the staged history after its
    // online pass.
    // this wave's share of the (staged part of the) history, into registers ahead of the barrier so
    // that it is not queued behind the row loads: positions c * 2048 + wave * 256 + q * 64 + lane;
    // unconditional loads over a zero-size range when penalties are off
    constexpr int HQ = HSTAGE / (4 * NT);
    const int n_stage = (int)min<int64_t>(n_hist, HSTAGE);
    int hq[HQ * 4];
    {
      const uint64_t hb = reinterpret_cast<uint64_t>(a.prm.hist_ids + (R.pen_on ? R.h_lo : 0));
      const uint32_t hb_lo = __builtin_amdgcn_readfirstlane((uint32_t)hb);
      const uint32_t hb_hi = __builtin_amdgcn_readfirstlane((uint32_t)(hb >> 32));
      const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<void*>(((uint64_t)hb_hi << 32) | hb_lo), (short)0,
          __builtin_amdgcn_readfirstlane(R.pen_on ? n_stage * 4 : 0), 0x00020000);
      const int hoff = (wave_id() * 256 + lane_id()) * 4;
#pragma unroll
      for (int t = 0; t < HQ * 4; ++t)
        hq[t] = __builtin_amdgcn_raw_buffer_load_b32(hrs, hoff + ((t >> 2) * 2048 + (t & 3) * 64) * 4, 0, 0);
    }
    if (threadIdx.x == 0) {
      s.ready = 0;
      s.n_list = 0;
      s.fxsum = 0;
      s.flags = 0;
    }
    if (threadIdx.x < 256) {
      s.kh_cnt[threadIdx.x] = 0u;
      s.kh_min[threadIdx.x] = 0xffffffffu;
    }
    if (R.pen_on) {
      uint4* bm4 = reinterpret_cast<uint4*>(s.bitmap);
      for (int i = threadIdx.x; i < NWORDS / 4; i += NT) bm4[i] = make_uint4(0u, 0u, 0u, 0u);
    }
    __syncthreads();  // LDS of the previous row is no longer in use; per-row LDS state is cleared
    // the rest of the pipeline's first slots
    static_for<PIPE - PIPE0>([&](auto jc) __attribute__((always_inline)) {
      issue(std::integral_constant<int, decltype(jc)::value + PIPE0>{});
    });
    if (R.pen_on) {
      int32_t* hst = hist_stage(s);
      uint32_t bad = 0;
#pragma unroll
      for (int t = 0; t < HQ * 4; ++t) {
        const int i = (t >> 2) * 2048 + wave_id() * 256 + (t & 3) * 64 + lane_id();
        if (i < n_stage) {
          const int id = hq[t];
          if ((unsigned)id >= (unsigned)R.V) {
            bad = FLAG_BAD_INPUT;
          } else {
            const int code = body_code<DT>(R, id);
            if (code >= 0) atomicOr(&s.bitmap[code >> 5], 1u << (code & 31));
          }
          hst[i] = id;
        }
      }
      bad = wave_or(bad);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");  // LDS only: row loads stay in flight
      if (lane_id() == 0) {
        if (bad) atomicOr(&s.flags, bad);
        atomicAdd(&s.ready, 1u);
      }
    }
    if (builder) {
      if (R.pen_on) wait_ready(s, (uint32_t)NW);
      const uint32_t bflags0 = finish_presence<DT>(s, R, a.prm.hist_ids);
      build_ranks<DT>(s, R, a.prm.hist_ids, bflags0);
    }
    const int jfull = __builtin_amdgcn_readfirstlane(nslots / NT);  // slots 0..jfull-1 all live
    if (R.pen_on) wait_ready(s, (uint32_t)NW + 1u);  // the masks below need the finished bitmap

    // ---------------- online max / sum-exp over the registers ----------------
    // The reference starts finite: a -inf element then gives exp2(-inf) = 0 rather than NaN, and the
    // first finite slot always moves the reference before anything is accumulated against it.
    // Maxima are taken over the products x r (the processed logits before the +0 that canonicalises
    // -0), which the sums need anyway; being results of arithmetic they need no quieting before a
    // max.  fl(x r) is monotone in x, so these are the products of the x maxima.
    float xm = -INFINITY, mref = MREF0;  // xm: this thread's maximum product
    // The thread's best slot pair so far (its data, pair index; xm is its maximum) and the largest
    // maximum of its other pairs: the gather tests the best pair from this copy, and only a thread
    // whose other pairs may reach the bound goes through the slot-by-slot pass.
    uint4 bd0 = make_uint4(DT::NEG, DT::NEG, DT::NEG, DT::NEG), bd1 = bd0;
    int bj = 0;
    float b2 = -INFINITY;
    float acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, acc3 = 0.f;
    const float rr = R.r;
    // the reference moves when a pair maximum gives z L2E above mref + 32; zthr is that point in z
    // units lowered by one (log2) unit, a cheap filter in front of the exact test
    constexpr float INV_L2E = 0.693147180559945309f;
    float zthr = (mref + 31.0f) * INV_L2E;
    // the -inf pattern in a register, so that masking is one bit-select per word
    uint32_t neg;
    asm volatile("s_mov_b32 %0, %1" : "=s"(neg) : "i"(DT::NEG));
    // Penalised rows with short histories count them in the middle of the online pass and load the
    // original value of each first occurrence there, so the loads complete under the stream; the
    // values are staged in LDS after the pass.  (The original of a penalised element is its raw
    // logit, which the registers hold only masked.)
    constexpr int PCOUNT = J / 4;  // pair at which the count runs
    const bool count_early = R.pen_on && n_hist <= 4 * NT;
    int fid[4] = {0, 0, 0, 0};
    float fv[4];
    // slots are taken in pairs: one reference test and one running-maximum update per pair
    static_for<J / 2>([&](auto pc) __attribute__((always_inline)) {
      constexpr int j0 = 2 * decltype(pc)::value;
      if constexpr (j0 / 2 == PCOUNT) {
        if (count_early) {
          wait_ready(s, (uint32_t)NW + 2u);
          const int32_t* hst = hist_stage(s);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int i = (int)threadIdx.x + q * NT;
            const int id = i < (int)n_hist ? hst[i] : -1;
            const int u = (unsigned)id < (unsigned)R.V ? extras_index<DT>(s, R, id) : -1;
            uint32_t first = 0xffffu;
            if (u >= 0) {
              if (atomicAdd(&s.x_cnt[u], 1u) == 0u) first = (uint32_t)u;
              s.x_pos[u] = id;  // every counting thread of this id writes the same value
            }
            s.first_u[q * NT + threadIdx.x] = (uint16_t)first;
            fid[q] = first != 0xffffu ? id : 0;
          }
        }
        // unconditional loads: a load under a branch is merged at its join, which waits for it
#pragma unroll
        for (int q = 0; q < 4; ++q) fv[q] = load_pos<DT>(R, fid[q]);
      }
      if constexpr (j0 + PIPE < J) issue(std::integral_constant<int, j0 + PIPE>{});
      if constexpr (j0 + 1 + PIPE < J) issue(std::integral_constant<int, j0 + 1 + PIPE>{});
      float v[2][DT::VEC], sm[2];
      uint4 dc[2];
      static_for<2>([&](auto hc) __attribute__((always_inline)) {
        constexpr int h = decltype(hc)::value;
        constexpr int j = j0 + h;
        // only slots at or past JLO can be partly filled (the host picks J so that the first JLO
        // slots of every thread are live)
        if constexpr (j >= JLO) {
          if (j >= jfull) {  // wave-uniform: the partly filled tail slots
            const bool dead = j * NT + (int)threadIdx.x >= nslots;
            uint4 dj = ch.template get<j>();
            dj.x = dead ? DT::NEG : dj.x;
            dj.y = dead ? DT::NEG : dj.y;
            dj.z = dead ? DT::NEG : dj.z;
            dj.w = dead ? DT::NEG : dj.w;
            ch.template set<j>(dj);
          }
        }
        if (R.pen_on) {
          const int sl = j * NT + threadIdx.x;
          const uint32_t byte = (s.bitmap[sl >> 2] >> ((sl & 3) * 8)) & 255u;
          const uint4 mk = s.masktab[byte];
          uint4 dj = ch.template get<j>();
          dj.x = (neg & mk.x) | (dj.x & ~mk.x);
          dj.y = (neg & mk.y) | (dj.y & ~mk.y);
          dj.z = (neg & mk.z) | (dj.z & ~mk.z);
          dj.w = (neg & mk.w) | (dj.w & ~mk.w);
          ch.template set<j>(dj);
        }
        const uint4 dcur = ch.template get<j>();
        dc[h] = dcur;
#pragma unroll
        for (int e = 0; e < DT::VEC; ++e) v[h][e] = DT::get(dcur, e) * rr;
        float mx = v[h][0];
#pragma unroll
        for (int e = 1; e < DT::VEC; ++e) mx = fmaxf(mx, v[h][e]);
        sm[h] = mx;
      });
      const float pm = fmaxf(sm[0], sm[1]);
      {
        const bool nb = pm > xm;  // ties keep the earlier pair and count toward b2
        const float t = nb ? xm : pm;
        b2 = t > b2 ? t : b2;
        xm = nb ? pm : xm;
        bj = nb ? j0 / 2 : bj;
        bd0.x = nb ? dc[0].x : bd0.x;
        bd0.y = nb ? dc[0].y : bd0.y;
        bd0.z = nb ? dc[0].z : bd0.z;
        bd0.w = nb ? dc[0].w : bd0.w;
        bd1.x = nb ? dc[1].x : bd1.x;
        bd1.y = nb ? dc[1].y : bd1.y;
        bd1.z = nb ? dc[1].z : bd1.z;
        bd1.w = nb ? dc[1].w : bd1.w;
        // keep the updates here: left to itself the compiler sinks them into the gather, keeping
        // every pair maximum live (and spilled) across the reduction
        asm volatile("" : "+v"(b2), "+v"(xm), "+v"(bj), "+v"(bd0.x), "+v"(bd0.y), "+v"(bd0.z), "+v"(bd0.w),
                     "+v"(bd1.x), "+v"(bd1.y), "+v"(bd1.z), "+v"(bd1.w));
      }
      // 16-bit slot-maximum codes, two per word (slot-pair-major)
      if constexpr (j0 + 1 < J)
        s.scode[(j0 / 2) * NT + threadIdx.x] = __builtin_amdgcn_perm(f2key(sm[1]), f2key(sm[0]), 0x07060302u);
      // sums run over the canonical z = fl32(x r) (exactly what the logprobs are defined on), as
      // 2^(z L2E - mref) with a reference mref in log2 units
      if (pm > zthr) {
        const float sref = pm * L2E;
        if (sref > mref + 32.0f) {  // move the reference lazily: exp2 arguments stay below 32
          const float f = __builtin_amdgcn_exp2f(mref - sref);
          acc0 *= f;
          acc1 *= f;
          acc2 *= f;
          acc3 *= f;
          mref = sref;
          zthr = (mref + 31.0f) * INV_L2E;
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < DT::VEC; e += 4) {
          acc0 += __builtin_amdgcn_exp2f(__builtin_fmaf(v[h][e + 0], L2E, -mref));
          acc1 += __builtin_amdgcn_exp2f(__builtin_fmaf(v[h][e + 1], L2E, -mref));
          acc2 += __builtin_amdgcn_exp2f(__builtin_fmaf(v[h][e + 2], L2E, -mref));
          acc3 += __builtin_amdgcn_exp2f(__builtin_fmaf(v[h][e + 3], L2E, -mref));
        }
    });
    float ssum = (acc0 + acc1) + (acc2 + acc3);

    // this thread's share of the staged history into the counts (read after the barrier below),
    // unless counted in the pass; the originals of the extras entries into LDS where all of them are
    // known here (rows without penalties, and rows counted in the pass)
    if (R.pen_on && n_hist <= HSTAGE && !count_early) {
      wait_ready(s, (uint32_t)NW + 2u);
      const int32_t* hst = hist_stage(s);
      for (int i = threadIdx.x; i < (int)n_hist; i += NT) count_history_id<DT>(s, R, hst[i]);
    }
    const bool staged = !R.pen_on || count_early;
    if (count_early) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t u = s.first_u[q * NT + threadIdx.x];
        if (u != 0xffffu) s.x_val[u] = fv[q];
      }
    }
    if (staged && (int)threadIdx.x < n_ht0) s.x_val[(R.pen_on ? s.n_body : 0) + (int)threadIdx.x] = xht;

    // maximum of this thread's register elements (a subset of the row, so the K-th largest of these
    // per-thread maxima bounds the K-th largest z of the row from below; K covers top-k and top-n)
    const float tmax_z = xm + 0.0f;  // canonical (-0 -> +0)
    int Ksel = R.k_on ? R.k : 0;
    if (a.mode == 0 && a.n_top > Ksel) Ksel = a.n_top;
    const bool want_kth = Ksel > 0 && Ksel <= NT;

    // ---------------- workgroup reduction ----------------
    // Barrier A publishes every wave's partials (the history counts are complete then too), B the
    // extras' maxima and the K-th bound histogram, C (rows with extras only) the extras' mass.  Every
    // thread combines the partials in the same fixed order, so all hold identical row statistics.
    {
      const float wm = wave_max(mref);
      const float wsum = wave_sum(ssum * rel2(mref, wm));
      const float wxm = wave_max(xm);
      const bool tv = tmax_z > -INFINITY;
      const float thi = wave_max(tv ? tmax_z : -INFINITY);
      const float tlo = wave_min(tv ? tmax_z : INFINITY);
      if (lane_id() == 0) {
        const int w = wave_id();
        s.wp[0][w] = wm;
        s.wp[1][w] = wsum;
        s.wp[2][w] = wxm;
        s.wp[3][w] = thi;
        s.wp[4][w] = tlo;
      }
    }
    __syncthreads();  // A
    clear_count_arrays(s);  // totals of the counting resolver (read after barrier D)
    float bm = s.wp[0][0], bs = s.wp[1][0], bxm = s.wp[2][0], thi = s.wp[3][0], tlo = s.wp[4][0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      lse_combine(bm, bs, s.wp[0][w], s.wp[1][w]);
      bxm = fmaxf(bxm, s.wp[2][w]);
      thi = fmaxf(thi, s.wp[3][w]);
      tlo = fminf(tlo, s.wp[4][w]);
    }
    if (want_kth && thi > -INFINITY && tmax_z > -INFINITY) {
      const float width = thi - tlo;
      const float scale = (width > 0.0f && width < INFINITY) ? 256.0f / width : 0.0f;
      const float f = (tmax_z - tlo) * scale;
      const int b = f >= 255.0f ? 255 : (f > 0.0f ? (int)f : 0);
      atomicAdd(&s.kh_cnt[b], 1u);
      atomicMin(&s.kh_min[b], f2key(tmax_z));
    }
    // extras: originals from memory with their penalties, entered into the row sum through an
    // order-independent fixed-point sum
    int n_ext = 0;
    float xmx = -INFINITY;
    if (extras_any) {
      n_ext = s.n_ext;
      uint32_t myflags = 0;
      for (int xi0 = threadIdx.x; xi0 < n_ext; xi0 += 4 * NT) {
        int idv[4];
        float xv[4];
        if (staged) {  // originals staged in LDS before the barrier
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int xi = xi0 + q * NT;
            xv[q] = xi < n_ext ? s.x_val[xi] : 0.f;
          }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {  // all loads in flight before the first use
            const int xi = xi0 + q * NT;
            const int pq = xi < n_ext ? s.x_pos[xi] : 0;
            idv[q] = (unsigned)pq < (unsigned)R.V ? pq : 0;  // defensive: only in-row reads
            xv[q] = load_pos<DT>(R, idv[q]);
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int xi = xi0 + q * NT;
          if (xi < n_ext) {
            const uint32_t cnt = s.x_cnt[xi];
            float x = xv[q];
            if (cnt > 0) x = penalise(x, cnt, R.rep, R.freq, R.pres);
            s.x_val[xi] = x;
            xmx = fmaxf(xmx, x);
            if (x != x) myflags |= FLAG_BAD_INPUT;
          }
        }
      }
      if (myflags) atomicOr(&s.flags, myflags);
      const float wx = wave_max(xmx);
      if (lane_id() == 0) s.wp[5][wave_id()] = wx;
    }
    __syncthreads();  // B
    uint32_t ext_flags = 0;
    float eref = bm;
    if (extras_any) {
      ext_flags = s.flags;
      float bxx = s.wp[5][0];
#pragma unroll
      for (int w = 1; w < NW; ++w) bxx = fmaxf(bxx, s.wp[5][w]);
      bxm = fmaxf(bxm, bxx * rr);  // the extras' maximum as a product
      // reference for the extras: at or above every extras term, so each term is <= 1
      eref = fmaxf(bm, (bxx * rr) * L2E);
      uint64_t fx = 0;
      for (int xi = threadIdx.x; xi < n_ext; xi += NT)
        fx += fixmass(__builtin_amdgcn_exp2f(__builtin_fmaf(s.x_val[xi] * rr, L2E, -eref)));
      fx = wave_sum_u64(fx);
      if (lane_id() == 0 && fx) atomicAdd(reinterpret_cast<unsigned long long*>(&s.fxsum), (unsigned long long)fx);
    }
    const float beta_sel = (want_kth && thi > -INFINITY) ? kth_from_hist(s, Ksel) : -INFINITY;
    // The extras' mass joins the row sum behind barrier C only where something before the gather
    // needs the sum (the chunk exchange, the top-p-only bound); otherwise after barrier D.
    const bool fx_late = extras_any && !(P > 1 || (!R.greedy && !R.k_on && !R.minp_on && R.topp_on));
    auto fold_extras = [&](float& m2, float& s2) {
      const uint64_t fx = s.fxsum;
      if (eref > m2) {
        s2 = s2 * rel2(m2, eref);
        m2 = eref;
      }
      s2 += (float)((double)fx / FIX_SCALE) * rel2(eref, m2);
    };
    if (extras_any && !fx_late) {
      __syncthreads();  // C
      fold_extras(bm, bs);
    }
    const uint32_t bflags = R.flags | ext_flags;

    // ---------------- combine the chunks of the row (fixed chunk order) ----------------
    float row_xm = bxm, row_mref = bm, row_s = bs, row_beta = beta_sel;
    uint32_t row_flags = bflags;
    if (P > 1) {
      if (threadIdx.x == 0) {
        st_agent(&X.gstats[c].xm, bxm);
        st_agent(&X.gstats[c].mref, bm);
        st_agent(&X.gstats[c].s, bs);
        st_agent(&X.gstats[c].flags, bflags);
        st_agent(&X.gstats[c].beta_sel, beta_sel);
      }
      group_barrier(X.gsync, P);
      row_xm = -INFINITY;
      row_mref = -INFINITY;
      row_s = 0.f;
      row_beta = -INFINITY;
      row_flags = 0;
      for (int q = 0; q < P; ++q) {
        row_xm = fmaxf(row_xm, ld_agent(&X.gstats[q].xm));
        lse_combine(row_mref, row_s, ld_agent(&X.gstats[q].mref), ld_agent(&X.gstats[q].s));
        row_beta = fmaxf(row_beta, ld_agent(&X.gstats[q].beta_sel));
        row_flags |= ld_agent(&X.gstats[q].flags);
      }
    }

    // ---------------- row statistics ----------------
    const float m = row_xm + 0.0f;  // the maxima are products already
    X.m = m;
    X.row_beta = row_beta;
    X.n_ext = n_ext;
    if (!(m > -INFINITY)) row_flags |= FLAG_EMPTY;
    const bool bad_vals = (m == INFINITY) || isnan(row_s) || isnan(m);
    if (bad_vals) row_flags |= FLAG_BAD_INPUT;
    const bool skip = (row_flags & FLAG_EMPTY) || bad_vals;

    // ---------------- candidate bound ----------------
    X.tau_m = R.minp_on ? __fadd_rn(m, log_minp_of(R.minp)) : -INFINITY;
    float beta_S = -INFINITY;
    if (R.greedy) {
      beta_S = m;
    } else if (R.k_on || R.minp_on) {
      beta_S = fmaxf(R.k_on ? row_beta : -INFINITY, X.tau_m);
    } else if (R.topp_on && R.p <= 0.9999f && !skip) {
      beta_S = topp_bound(row_mref, row_s, m, R.p, R.V);
    }
    float beta_list = beta_S;
    if (a.mode == 0 && a.n_top > 0) beta_list = fminf(beta_list, row_beta);
    const bool no_bound = !(beta_list > -INFINITY);

    // ---------------- gather candidates z >= beta_list into the LDS list ----------------
    // (the list counter was cleared at the start of the row)
    if (!skip && !no_bound) {
      const float r = R.r;
      const float bl = beta_list;
      // a candidate is an element whose product x r is >= bl (canon only turns -0 into +0)
      const int pos_t = R.head + (int)(R.s0 + threadIdx.x) * DT::VEC;
      // the best pair, from its register copy: one list claim per wave, each lane's place being its
      // exclusive prefix of the candidate counts
      {
        uint32_t cm = 0;  // bit e: element e of the pair (slot 2 bj, then 2 bj + 1)
#pragma unroll
        for (int e = 0; e < DT::VEC; ++e) {
          cm |= (canon(DT::get(bd0, e), r) >= bl ? 1u : 0u) << e;
          cm |= (canon(DT::get(bd1, e), r) >= bl ? 1u : 0u) << (DT::VEC + e);
        }
        const int c = __popc(cm);
        const int incl = wave_incl_scan_i(c);
        const int total = lane_i32(incl, 63);
        if (total > 0) {
          int base = 0;
          if (lane_id() == 0) base = atomicAdd(&s.n_list, total);
          int idx = __builtin_amdgcn_readfirstlane(base) + incl - c;
          const int pb = pos_t + 2 * bj * NT * DT::VEC;
          while (cm) {
            const int b = __ffs(cm) - 1;
            cm &= cm - 1;
            const int e = b % DT::VEC;
            const float x = b < DT::VEC ? DT::get(bd0, e) : DT::get(bd1, e);
            if (idx < LCAP) s.sk[idx] = cand_key(canon(x, r), pb + (b < DT::VEC ? 0 : NT * DT::VEC) + e);
            ++idx;
          }
        }
      }
      // the other pairs of threads whose second-best pair maximum reaches the bound: pass 1 from the
      // slot-maximum codes the online pass left in LDS (a code at or above the bound's code:
      // truncating a monotone key keeps smax >= bl => code(smax) >= code(bl)), pass 2 from the
      // registers
      const bool more = b2 >= bl;
      if (__ballot(more)) {
        const uint32_t tcode = f2key(bl) >> 16;
        // an opaque copy of the thread index, so that the code addresses are not shared with the
        // online pass's stores (which would keep them live, spilled, across the pass)
        int tid = (int)threadIdx.x;
        asm volatile("" : "+v"(tid));
        // per lane, the pairs other than its best whose larger slot code reaches the bound's code
        // (word i holds the codes of pair i); the wave takes their union
        uint32_t pm = 0;
        static_for<J / 2>([&](auto ic) __attribute__((always_inline)) {
          constexpr int i = decltype(ic)::value;
          const uint32_t w = s.scode[i * NT + tid];
          pm |= (max(w & 0xffffu, w >> 16) >= tcode ? 1u : 0u) << i;
        });
        pm = more ? pm & ~(1u << bj) : 0u;
        uint32_t wpm = wave_or(pm);
        // one pair at a time, picked from the registers by its run-time index; the lanes that flagged
        // it mark their candidates in a bit mask and the wave takes one list claim
        while (wpm) {
          const int i = __builtin_ctz(wpm);
          wpm &= wpm - 1;
          const uint4 p0 = ch.pick(2 * i), p1 = ch.pick(2 * i + 1);
          const bool use = (pm >> i) & 1u;
          uint32_t cm = 0;  // bit e: element e of the pair (slot 2 i, then 2 i + 1)
#pragma unroll
          for (int e = 0; e < DT::VEC; ++e) {
            cm |= (use && canon(DT::get(p0, e), r) >= bl ? 1u : 0u) << e;
            cm |= (use && canon(DT::get(p1, e), r) >= bl ? 1u : 0u) << (DT::VEC + e);
          }
          const int c = __popc(cm);
          const int incl = wave_incl_scan_i(c);
          const int total = lane_i32(incl, 63);
          if (total > 0) {
            int base = 0;
            if (lane_id() == 0) base = atomicAdd(&s.n_list, total);
            int idx = __builtin_amdgcn_readfirstlane(base) + incl - c;
            const int pp = pos_t + 2 * i * NT * DT::VEC;
            while (cm) {
              const int b = __ffs(cm) - 1;
              cm &= cm - 1;
              const int e = b % DT::VEC;
              const float x = b < DT::VEC ? DT::get(p0, e) : DT::get(p1, e);
              if (idx < LCAP) s.sk[idx] = cand_key(canon(x, r), pp + (b < DT::VEC ? 0 : NT * DT::VEC) + e);
              ++idx;
            }
          }
        }
      }
      FOR_EXTRAS(s, n_ext, {
        const float z = canon(x, r);
        if (z >= bl) {
          const int idx = atomicAdd(&s.n_list, 1);
          if (idx < LCAP) s.sk[idx] = cand_key(z, pos);
        }
      })
    }
    __syncthreads();  // D
    if (fx_late) fold_extras(row_mref, row_s);  // P == 1 here: the row's own sums
    // the full-vocabulary normaliser in double, now that the row's registers are released
    {
      const RowDoubles RD = row_doubles(row_mref, row_s, m);
      X.L = RD.L;
      X.zfull = RD.zfull;
    }
    int n_list = s.n_list;
    bool overflow = !skip && (no_bound || n_list > LCAP || n_list == 0);
    if (P > 1) n_list = union_lists(s, R, X, n_list, overflow);
    X.n_list = n_list;

    // ---------------- resolution ----------------
    Resolution res;
    res.tau = INFINITY;
    res.zs = 0.f;
    res.zmin = -INFINITY;
    res.kept = 0;
    res.id = -1;
    res.zid = -INFINITY;
    res.id_here = leader;
    const OutArgs oa{a.mode, a.n_top, a.V, a.out_top_ids, a.out_top_logprobs, a.out_probs};
    if (skip) {
      // empty row or NaN / +inf values: nothing to resolve
    } else if (!overflow) {
      if (leader) {
        if (X.n_list <= SMALL_LIST) {
          res = resolve_count(oa, s, R, X, res);  // every thread holds the result
        } else {
          res = resolve_list(oa, s, R, X, res);
        }
      }
    } else {
      res = resolve_general<DT>(oa, s, R, X, res);
    }

    // ---------------- per-row outputs ----------------
    if (a.mode == 0) {
      if (skip) {
        if (leader) {
          if (threadIdx.x == 0) {
            a.out_ids[row] = -1;
            a.out_logprobs[row] = -INFINITY;
          }
          for (int t = threadIdx.x; t < a.n_top; t += NT) {
            a.out_top_ids[row * a.n_top + t] = -1;
            a.out_top_logprobs[row * a.n_top + t] = -INFINITY;
          }
        }
      } else if (res.id_here && threadIdx.x == 0) {
        a.out_ids[row] = res.id;
        a.out_logprobs[row] = res.id >= 0 ? (float)((double)res.zid - (double)m - X.L) : -INFINITY;
      }
      // early-feedback backfill into the next iteration's token slots (an empty row sends -1)
      if (a.next_tokens && threadIdx.x == 0 && (skip ? leader : res.id_here)) {
        const int32_t d = a.backfill_dest[row];
        if (d >= 0 && (int64_t)d < a.next_len) a.next_tokens[d] = skip ? -1 : res.id;
      }
    }
    if (leader && threadIdx.x == 0) {
      if (MULTI && __hip_atomic_load(&X.gsync->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
        row_flags |= FLAG_TIMEOUT;
      if (a.out_flags) a.out_flags[row] = row_flags;
      if (a.mode == 1) {
        if (a.out_threshold) a.out_threshold[row] = skip ? -INFINITY : res.zmin;
        if (a.out_kept) a.out_kept[row] = skip ? 0 : res.kept;
        if (a.out_log_norm) a.out_log_norm[row] = skip ? -INFINITY : (float)((double)m + log((double)res.zs));
      }
    }
    if (a.mode == 1 && a.out_probs) dense_probs<DT>(oa, s, R, X, res, skip, P > 1 && !skip && !overflow);
    if (MULTI) __syncthreads();  // the next row reuses LDS
  }
}

// Single-chunk rows: one workgroup per row, no workspace.
template <class DT, int J, bool SEG>
__global__ __launch_bounds__(NT) void k_sample(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& s = *reinterpret_cast<Smem*>(smem_raw);
  if (threadIdx.x < 256) s.masktab[threadIdx.x] = DT::mask_of(threadIdx.x);
  RowCtx X;
  memset(&X, 0, sizeof X);
  process_row<DT, J, false, SEG>(a, s, X, (int64_t)blockIdx.x, 0);
}

// Rows of P > 1 chunks: a persistent cooperative grid of row groups; the P workgroups of a group
// process the group's rows in lockstep and exchange per-chunk results through the workspace.
template <class DT, int J, bool SEG>
__global__ __launch_bounds__(NT) void k_sample_multi(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& s = *reinterpret_cast<Smem*>(smem_raw);

  // block -> (group, chunk); with xcd_map the P chunks of a group sit on one XCD (consecutive
  // workgroups are dispatched round-robin over the 8 XCDs)
  int g, c;
  if (a.xcd_map) {
    const int b = blockIdx.x, xcd = b & 7, li = b >> 3;
    g = (li / a.P) * 8 + xcd;
    c = li % a.P;
  } else {
    g = blockIdx.x / a.P;
    c = blockIdx.x % a.P;
  }
  RowCtx X;
  memset(&X, 0, sizeof X);
  {
    unsigned char* wsg = a.ws + (int64_t)g * a.ws_group_bytes;
    const WsLayout WL(a.P);
    X.gsync = reinterpret_cast<GroupSync*>(wsg + WL.sync);
    X.gstats = reinterpret_cast<ChunkStats*>(wsg + WL.stats);
    X.gres = reinterpret_cast<GroupRes*>(wsg + WL.res);
    X.ghist = reinterpret_cast<uint64_t*>(wsg + WL.hist);
    X.glists = reinterpret_cast<uint64_t*>(wsg + WL.lists);
  }
  if (threadIdx.x < 256) s.masktab[threadIdx.x] = DT::mask_of(threadIdx.x);
  for (int64_t row = g; row < a.B; row += a.n_groups) process_row<DT, J, true, SEG>(a, s, X, row, c);

  // leave the group's counters at zero for the next call
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(&X.gsync->exit, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (old == (uint32_t)a.P - 1) {
      __hip_atomic_store(&X.gsync->arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&X.gsync->error, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&X.gsync->exit, 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

}  // namespace

// ==============================================================================================
// Standalone penalties: albireo_apply_penalties.  A workgroup handles one tile of one row: every id of
// the row's output history, prompt history or penalty state that falls in the tile is folded into a
// 32-bit word per tile element in LDS (bits 0-30 the output count, bit 31 the prompt mark: the penalty
// state's encoding), and the tile is streamed to the fp32 output (each element read and written by the
// same thread, so the output may alias an fp32 input).  The words are exact for any history length.
// ==============================================================================================
namespace {

constexpr int PEN_NT = 256;
constexpr int64_t PEN_TILE = 16384;  // elements per workgroup (64 KB of LDS words)

// The uniforms alone (one thread per row), for callers that sample elsewhere.
__global__ __launch_bounds__(256) void k_philox_uniforms(uint64_t seed, uint64_t step, const int64_t* seq_ids,
                                                         int64_t B, float* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < B) out[i] = philox_uniform(seed, step, seq_ids ? (uint64_t)seq_ids[i] : (uint64_t)i);
}

// The backfill alone (one thread per row).
__global__ __launch_bounds__(256) void k_backfill(const int32_t* ids, const int32_t* dest, int64_t B,
                                                  int32_t* next_tokens, int64_t next_len) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < B) {
    const int32_t d = dest[i];
    if (d >= 0 && (int64_t)d < next_len) next_tokens[d] = ids[i];
  }
}

// Zero n sixteen-byte words (grid-stride): restores the no-alloc scratch after a call whose launches
// the runtime refused part-way.
__global__ __launch_bounds__(256) void k_zero16(uint4* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = make_uint4(0, 0, 0, 0);
}

// The prompt history (repetition only) and the per-sequence penalty state, beside the output history.
struct PenExtra {
  const int64_t* prompt_offsets;
  const int32_t* prompt_ids;
  int64_t prompt_len;
  const int32_t* st_ids;
  const uint32_t* st_counts;
  const int32_t* st_len;
  int32_t st_cap;
};

template <class DT>
__global__ __launch_bounds__(PEN_NT) void k_penalties(const unsigned char* logits, int64_t V, int64_t ld,
                                                      DevParams prm, PenExtra ex, float* out) {
  __shared__ uint32_t cvs[PEN_TILE];
  const int64_t row = blockIdx.y;
  const int64_t t0 = (int64_t)blockIdx.x * PEN_TILE;
  const int64_t t1 = min(V, t0 + PEN_TILE);
  const unsigned char* rowp = logits + row * ld * DT::ES;
  float rep = prm.rep ? prm.rep[row] : 1.0f;
  float freq = prm.freq ? prm.freq[row] : 0.0f;
  float pres = prm.pres ? prm.pres[row] : 0.0f;
  if (!(rep > 0.0f) || isinf(rep)) rep = 1.0f;
  if (!isfinite(freq)) freq = 0.0f;
  if (!isfinite(pres)) pres = 0.0f;
  int64_t lo = 0, hi = 0;
  if (prm.hist_offsets) {
    lo = prm.hist_offsets[row];
    hi = prm.hist_offsets[row + 1];
    if (lo < 0 || hi < lo || hi > prm.hist_len) lo = hi = 0;
  }
  int64_t plo = 0, phi = 0;
  if (ex.prompt_offsets) {
    plo = ex.prompt_offsets[row];
    phi = ex.prompt_offsets[row + 1];
    if (plo < 0 || phi < plo || phi > ex.prompt_len) plo = phi = 0;
  }
  int sn = 0;
  if (ex.st_len) {
    sn = ex.st_len[row];
    sn = sn < 0 ? 0 : (sn > ex.st_cap ? ex.st_cap : sn);
  }
  const bool pen = hi > lo || phi > plo || sn > 0;
  if (pen) {
    for (int i = threadIdx.x; i < PEN_TILE; i += PEN_NT) cvs[i] = 0;
    __syncthreads();
    for (int64_t h = lo + threadIdx.x; h < hi; h += PEN_NT) {
      const int id = prm.hist_ids[h];
      if (id >= t0 && id < t1) atomicAdd(&cvs[id - t0], 1u);
    }
    for (int64_t h = plo + threadIdx.x; h < phi; h += PEN_NT) {
      const int id = ex.prompt_ids[h];
      if (id >= t0 && id < t1) atomicOr(&cvs[id - t0], 0x80000000u);
    }
    for (int e = threadIdx.x; e < sn; e += PEN_NT) {
      const int id = ex.st_ids[row * ex.st_cap + e];
      if (id >= t0 && id < t1) cvs[id - t0] = ex.st_counts[row * ex.st_cap + e];  // distinct ids
    }
    __syncthreads();
  }
  float* orow = out + row * V;
  for (int64_t i = t0 + threadIdx.x; i < t1; i += PEN_NT) {
    float x = DT::load1(rowp, i);
    if (pen) {
      const uint32_t cv = cvs[i - t0];
      if (cv != 0) x = penalise_cv(x, cv, rep, freq, pres);
    }
    orow[i] = x;
  }
}

// ==============================================================================================
// Host side: geometry, capacity, workspace, launch
// ==============================================================================================
struct KernelInfo {
  const void* fn;
  int J;
};

template <class DT, int J, bool SEG>
KernelInfo kinfo1(bool multi) {
  return {multi ? reinterpret_cast<const void*>(&k_sample_multi<DT, J, SEG>)
                : reinterpret_cast<const void*>(&k_sample<DT, J, SEG>),
          J};
}

template <class DT, int J>
KernelInfo kinfo(bool multi, bool seg) {
  return seg ? kinfo1<DT, J, true>(multi) : kinfo1<DT, J, false>(multi);
}

template <class DT>
KernelInfo pick_kernel(int64_t chunk_slots, bool multi, bool seg) {
  if (chunk_slots <= (int64_t)JSIZES[0] * NT) return kinfo<DT, JSIZES[0]>(multi, seg);
  if (chunk_slots <= (int64_t)JSIZES[1] * NT) return kinfo<DT, JSIZES[1]>(multi, seg);
  if (chunk_slots <= (int64_t)JSIZES[2] * NT) return kinfo<DT, JSIZES[2]>(multi, seg);
  return kinfo<DT, JSIZES[3]>(multi, seg);
}

struct Geometry {
  int P;
  int64_t chunk_slots;
  KernelInfo k;
  int n_groups;
  int64_t group_bytes;
  size_t smem;
  bool ok;
};

struct DeviceCaps {
  int cus = 0;
  int blocks_per_cu = 0;
};

// Per (device, kernel) launch setup, done once: the dynamic-LDS attribute and the occupancy that
// bounds the persistent grid.
constexpr int MAX_DEV = 64;
constexpr int MAX_FN = 64;
std::mutex g_caps_mu;
int g_cus[MAX_DEV];
const void* g_fn[MAX_DEV][MAX_FN];
int g_bpc[MAX_DEV][MAX_FN];

hipError_t device_caps(int dev, const void* fn, size_t smem, DeviceCaps& out) {
  std::lock_guard<std::mutex> lk(g_caps_mu);
  if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
  if (g_cus[dev] == 0) {
    hipDeviceProp_t p;
    hipError_t e = hipGetDeviceProperties(&p, dev);
    if (e != hipSuccess) return e;
    g_cus[dev] = p.multiProcessorCount;
  }
  out.cus = g_cus[dev];
  for (int i = 0; i < MAX_FN; ++i) {
    if (g_fn[dev][i] == fn) {
      out.blocks_per_cu = g_bpc[dev][i];
      return hipSuccess;
    }
    if (g_fn[dev][i] == nullptr) {
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
      if (e != hipSuccess) return e;
      int nb = 0;
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, NT, smem);
      if (e != hipSuccess) return e;
      g_fn[dev][i] = fn;
      g_bpc[dev][i] = nb;
      out.blocks_per_cu = nb;
      return hipSuccess;
    }
  }
  return hipErrorUnknown;
}

// The shape part of the geometry (chunks per row, register slots, kernel, whether the kernels apply),
// from V and dtype alone, with no runtime call.
void shape_geometry(int64_t V, albireo_dtype_t dtype, bool seg, Geometry& G) {
  memset(&G, 0, sizeof G);
  const int VEC = dtype == ALBIREO_BF16 ? BF16T::VEC : F32T::VEC;
  const int64_t max_body = V / VEC;
  int64_t P = (max_body + (int64_t)JMAX * NT - 1) / ((int64_t)JMAX * NT);
  if (P < 1) P = 1;
  if (P > MAXP) return;
  G.P = (int)P;
  G.chunk_slots = (max_body + P - 1) / P;
  G.k = dtype == ALBIREO_BF16 ? pick_kernel<BF16T>(G.chunk_slots, G.P > 1, seg)
                              : pick_kernel<F32T>(G.chunk_slots, G.P > 1, seg);
  // the single-chunk kernel skips the dead-slot test below live_slots_min(J) (always true for the
  // size pick_kernel chose; a build restricted to one size can miss it for small rows)
  G.ok = !(G.P == 1 && max_body - 1 < (int64_t)live_slots_min(G.k.J) * NT);
}

hipError_t make_geometry(int64_t B, int64_t V, albireo_dtype_t dtype, Geometry& G, bool seg = false) {
  shape_geometry(V, dtype, seg, G);
  if (!G.ok) return hipSuccess;
  G.smem = sizeof(Smem);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  DeviceCaps caps;
  e = device_caps(dev, G.k.fn, G.smem, caps);
  if (e != hipSuccess) return e;
  if (G.P == 1) {  // one workgroup per row, nothing in the workspace
    G.n_groups = (int)B;
    G.group_bytes = 0;
    return hipSuccess;
  }
  int64_t cap_groups = (int64_t)caps.cus * (caps.blocks_per_cu > 0 ? caps.blocks_per_cu : 1) / G.P;
  if (cap_groups < 1) cap_groups = 1;
  G.n_groups = (int)(B < cap_groups ? B : cap_groups);
  if (G.n_groups < 1) G.n_groups = 1;
  G.group_bytes = WsLayout(G.P).total;
  return hipSuccess;
}

size_t required_ws(const Geometry& G) { return (size_t)G.group_bytes * (size_t)G.n_groups; }

// Workspace of the register-resident kernels for (B, V, dtype), 0 when they do not apply.
size_t legacy_ws(int64_t B, int64_t V, albireo_dtype_t dtype) {
  Geometry G;
  if (make_geometry(B, V, dtype, G) != hipSuccess || !G.ok) return 0;
  return required_ws(G);
}

// A prompt history or a penalty state is read by the streaming kernels only.
bool needs_stream(const albireo_params_t* params) {
  return params && (params->prompt_offsets || params->state);
}

// Kernel choice by shape alone (host only, no runtime call), so that a row gets the same arithmetic in
// every layout and batch: a row that fits one workgroup's registers is sampled by that one workgroup
// (no global round trip between its phases); wider rows, and rows with a prompt history or a penalty
// state, go to the streaming kernels; the cooperative chunked kernel takes what the streaming kernels
// cannot index (B x chunks >= 2^31).  Every sampling entry point routes through this one decision.
albireo_route_t route_of(int64_t B, int64_t V, albireo_dtype_t dtype, const albireo_params_t* params, bool seg) {
  if (B < 0 || V <= 0 || V >= ((int64_t)1 << 31) - 16 || (dtype != ALBIREO_F32 && dtype != ALBIREO_BF16))
    return ALBIREO_ROUTE_NONE;
  const bool st = albireo_stream::supported(B > 0 ? B : 1, V, dtype);
  if (needs_stream(params)) return st ? ALBIREO_ROUTE_STREAM : ALBIREO_ROUTE_NONE;
  Geometry G;
  shape_geometry(V, dtype, seg, G);
  if (G.ok && G.P == 1) return ALBIREO_ROUTE_ONE_WORKGROUP;
  if (st) return ALBIREO_ROUTE_STREAM;
  return G.ok ? ALBIREO_ROUTE_COOPERATIVE : ALBIREO_ROUTE_NONE;
}

albireo_status_t launch_sample(const KArgs& a0, const Geometry& G, hipStream_t stream) {
  KArgs a = a0;
  a.P = G.P;
  a.n_groups = G.n_groups;
  a.chunk_slots = G.chunk_slots;
  a.ws_group_bytes = G.group_bytes;
  const int grid = G.n_groups * G.P;
  a.xcd_map = (G.P > 1 && grid % (8 * G.P) == 0) ? 1 : 0;
  void* args[] = {&a};
  hipError_t e;
  if (G.P == 1) {
    e = hipLaunchKernel(G.k.fn, dim3(grid), dim3(NT), args, G.smem, stream);
  } else {
    e = hipLaunchCooperativeKernel(G.k.fn, dim3(grid), dim3(NT), args, (unsigned int)G.smem, stream);
  }
  return e == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

DevParams dev_params(const albireo_params_t* p) {
  DevParams d;
  memset(&d, 0, sizeof d);
  if (!p) return d;
  d.temperature = p->temperature;
  d.top_k = p->top_k;
  d.top_p = p->top_p;
  d.min_p = p->min_p;
  d.rep = p->repetition_penalty;
  d.freq = p->frequency_penalty;
  d.pres = p->presence_penalty;
  d.hist_offsets = p->hist_offsets;
  d.hist_ids = p->hist_ids;
  d.hist_len = p->hist_len;
  return d;
}

albireo_status_t check_common(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                              const albireo_params_t* params) {
  if (dtype != ALBIREO_F32 && dtype != ALBIREO_BF16) return ALBIREO_E_INVALID;
  if (B < 0 || V <= 0 || ld < V) return ALBIREO_E_INVALID;
  if (V >= ((int64_t)1 << 31) - 16 || B >= ((int64_t)1 << 31)) return ALBIREO_E_UNSUPPORTED;
  if (B > 0 && !logits) return ALBIREO_E_INVALID;
  const int es = dtype == ALBIREO_BF16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(logits) % es) return ALBIREO_E_INVALID;
  if (params && params->hist_offsets) {
    if (params->hist_len < 0) return ALBIREO_E_INVALID;
    if (params->hist_len > 0 && !params->hist_ids) return ALBIREO_E_INVALID;
  }
  if (params && params->prompt_offsets) {
    if (params->prompt_len < 0) return ALBIREO_E_INVALID;
    if (params->prompt_len > 0 && !params->prompt_ids) return ALBIREO_E_INVALID;
  }
  if (params && params->state) {
    const albireo_penalty_state_t* st = params->state;
    if (params->hist_offsets || params->prompt_offsets) return ALBIREO_E_INVALID;
    if (st->cap < 1 || st->cap > ALBIREO_MAX_STATE_ENTRIES) return ALBIREO_E_INVALID;
    if (B > 0 && (!st->ids || !st->counts || !st->len || !st->flags)) return ALBIREO_E_INVALID;
  }
  return ALBIREO_OK;
}

albireo_status_t check_ws(void* ws, size_t bytes, size_t need) {
  if (need == 0) return ALBIREO_OK;
  if (!ws || reinterpret_cast<uintptr_t>(ws) % 256) return ALBIREO_E_WORKSPACE;
  if (bytes < need) return ALBIREO_E_WORKSPACE;
  return ALBIREO_OK;
}

// The blocked (all-to-all receive) layout: checks that need no device.
albireo_status_t check_shards(const void* logits, albireo_dtype_t dtype, int64_t V, int64_t ld,
                              const albireo_shards_t& sh) {
  const int64_t es = dtype == ALBIREO_BF16 ? 2 : 4;
  const int64_t L = sh.shard_len, S = sh.shard_stride;
  if (L <= 0 || S < 0 || ld < 0) return ALBIREO_E_INVALID;
  if (ld < (L < V ? L : V)) return ALBIREO_E_INVALID;
  const int64_t t = (V + L - 1) / L;
  if (t > 1 && S < L) return ALBIREO_E_INVALID;  // blocks of one row must not overlap
  // every 16-byte slot inside one block: aligned base, row stride, block stride and block length
  if (reinterpret_cast<uintptr_t>(logits) % 16 || (L * es) % 16 || (S * es) % 16 || (ld * es) % 16)
    return ALBIREO_E_UNSUPPORTED;
  if (L * es / 16 > ((int64_t)1 << 31) || (t > 1 && (S - L) * es > ((int64_t)1 << 31))) return ALBIREO_E_UNSUPPORTED;
  return ALBIREO_OK;
}

// The blocked layout's kernel arguments (after check_shards), once the kernel size is known.
albireo_status_t shard_args(albireo_dtype_t dtype, int64_t V, const albireo_shards_t& sh, const Geometry& G,
                            KArgs& a) {
  const int64_t es = dtype == ALBIREO_BF16 ? 2 : 4;
  const int64_t L = sh.shard_len, S = sh.shard_stride;
  const int64_t t = (V + L - 1) / L;
  const int64_t sps = L * es / 16;
  const int64_t gap = t > 1 ? (S - L) * es : 0;
  // the lane offsets of all J slots a workgroup issues stay below 2^31
  const int64_t issued = (int64_t)G.k.J * NT;
  if (issued * 16 + (issued / sps + 1) * gap >= ((int64_t)1 << 31)) return ALBIREO_E_UNSUPPORTED;
  a.seg_sps = (uint32_t)sps;
  a.seg_magic = (uint32_t)(0xffffffffull / (uint64_t)sps);
  a.seg_ntq = (uint32_t)(NT / sps);
  a.seg_ntr = (uint32_t)(NT % sps);
  a.seg_gap = gap;
  return ALBIREO_OK;
}

// albireo_sample / albireo_sample_step / albireo_sample_sharded: shards NULL is the row-major layout;
// exactly one of uniforms and step is given.
albireo_status_t sample_impl(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                             const albireo_shards_t* shards, const albireo_params_t* params, const float* uniforms,
                             const albireo_step_t* step, int32_t* out_ids, float* out_logprobs, int32_t n_top,
                             int32_t* out_top_ids, float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  // the row-major checks; the blocked layout has its own stride rules (below)
  albireo_status_t st = check_common(logits, dtype, B, V, shards ? V : ld, params);
  if (st != ALBIREO_OK) return st;
  if (n_top < 0 || n_top > ALBIREO_MAX_TOP_N) return ALBIREO_E_INVALID;
  if (step && step->next_tokens && (!step->backfill_dest || step->next_len < 0)) return ALBIREO_E_INVALID;
  if (B == 0) return ALBIREO_OK;
  if ((!uniforms && !step) || !out_ids || !out_logprobs) return ALBIREO_E_INVALID;
  if (n_top > 0 && (!out_top_ids || !out_top_logprobs)) return ALBIREO_E_INVALID;
  if (shards) {
    st = check_shards(logits, dtype, V, ld, *shards);
    if (st != ALBIREO_OK) return st;
  }
  const albireo_route_t route = route_of(B, V, dtype, params, shards != nullptr);
  if (route == ALBIREO_ROUTE_NONE) return ALBIREO_E_UNSUPPORTED;
  if (route != ALBIREO_ROUTE_STREAM) {
    // the register-resident kernels
    Geometry G;
    if (make_geometry(B, V, dtype, G, shards != nullptr) != hipSuccess) return ALBIREO_E_LAUNCH;
    if (!G.ok) return ALBIREO_E_UNSUPPORTED;
    KArgs a;
    memset(&a, 0, sizeof a);
    if (shards) {
      st = shard_args(dtype, V, *shards, G, a);
      if (st != ALBIREO_OK) return st;
    }
    st = check_ws(workspace, workspace_bytes, required_ws(G));
    if (st != ALBIREO_OK) return st;
    a.logits = static_cast<const unsigned char*>(logits);
    a.B = B;
    a.V = V;
    a.ld = ld;
    a.prm = dev_params(params);
    a.uniforms = uniforms;
    if (step) {
      a.rng_on = 1;
      a.rng_seed = step->seed;
      a.rng_step = step->step;
      a.seq_ids = step->seq_ids;
      a.next_tokens = step->next_tokens;
      a.backfill_dest = step->backfill_dest;
      a.next_len = step->next_len;
    }
    a.out_ids = out_ids;
    a.out_logprobs = out_logprobs;
    a.n_top = n_top;
    a.out_top_ids = out_top_ids;
    a.out_top_logprobs = out_top_logprobs;
    a.out_flags = out_flags;
    a.mode = 0;
    a.ws = static_cast<unsigned char*>(workspace);
    return launch_sample(a, G, stream);
  }
  // the streaming kernels; their part of the workspace follows the register-resident kernels' part
  const size_t off = (size_t)align256((int64_t)legacy_ws(B, V, dtype));
  st = check_ws(workspace, workspace_bytes, off + albireo_stream::workspace_bytes(B, V, dtype));
  if (st != ALBIREO_OK) return st;
  albireo_stream::Request r;
  r.logits = logits;
  r.dtype = dtype;
  r.B = B;
  r.V = V;
  r.ld = ld;
  r.params = params;
  r.uniforms = uniforms;
  r.step = step;
  r.shards = shards;
  r.out_ids = out_ids;
  r.out_logprobs = out_logprobs;
  r.n_top = n_top;
  r.out_top_ids = out_top_ids;
  r.out_top_logprobs = out_top_logprobs;
  r.out_flags = out_flags;
  r.ws = static_cast<unsigned char*>(workspace) + off;
  r.stream = stream;
  return albireo_stream::launch(r);
}

}  // namespace

// ----------------------------------------------------------------------------------------------
// Device scratch of albireo_sample_noalloc: one array in every device's copy of the code object, held
// until the process ends.  In host code its name is only a host-side stand-in: the device address of
// each device's copy comes from hipGetSymbolAddress (once per device, with that device current) and
// only that address is ever passed to a kernel.
// ----------------------------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[ALBIREO_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[SCRATCH_DEVICES];   // per device: the address of its copy of `scratch`
bool g_scratch_dirty[SCRATCH_DEVICES];  // per device: a call returned ALBIREO_E_LAUNCH since the last fill

// The current device's scratch address (looked up on the first call on that device) and index.
albireo_status_t scratch_for_current_device(void** out, int* dev_out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_DEVICES) return ALBIREO_E_LAUNCH;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return ALBIREO_E_LAUNCH;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  *dev_out = dev;
  return ALBIREO_OK;
}
}  // namespace

extern "C" {

albireo_route_t albireo_sample_route(int64_t B, int64_t V, albireo_dtype_t dtype, const albireo_params_t* params,
                                    int32_t sharded) {
  return route_of(B, V, dtype, params, sharded != 0);
}

size_t albireo_workspace_size(int64_t B, int64_t V, albireo_dtype_t dtype, int32_t n_top) {
  (void)n_top;
  if (B <= 0 || V <= 0 || (dtype != ALBIREO_F32 && dtype != ALBIREO_BF16)) return 256;
  if (V >= ((int64_t)1 << 31) - 16) return 0;
  // the register-resident kernels' part, then the streaming kernels' part whenever they can serve the
  // shape (rows with a prompt history or a penalty state go to them whatever their width)
  const size_t legacy = legacy_ws(B, V, dtype);
  const size_t stream = albireo_stream::workspace_bytes(B, V, dtype);
  if (stream == 0) {
    Geometry G;
    if (make_geometry(B, V, dtype, G) != hipSuccess || !G.ok) return 0;
  }
  const size_t need = (size_t)align256((int64_t)legacy) + stream;
  return need < 256 ? 256 : need;
}

albireo_status_t albireo_sample(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                const albireo_params_t* params, const float* uniforms, int32_t* out_ids,
                                float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
  return sample_impl(logits, dtype, B, V, ld, nullptr, params, uniforms, nullptr, out_ids, out_logprobs, n_top,
                     out_top_ids, out_top_logprobs, out_flags, workspace, workspace_bytes, stream);
}

albireo_status_t albireo_sample_noalloc(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V,
                                        int64_t ld, const albireo_params_t* params, const float* uniforms,
                                        int32_t* out_ids, float* out_logprobs, int32_t n_top,
                                        int32_t* out_top_ids, float* out_top_logprobs, uint32_t* out_flags,
                                        hipStream_t stream) {
  // the same checks as albireo_sample decide the shape's validity; here only the scratch bound
  if (B > 0 && V > 0 && (dtype == ALBIREO_F32 || dtype == ALBIREO_BF16) &&
      albireo_workspace_size(B, V, dtype, n_top) > (size_t)ALBIREO_NOALLOC_SCRATCH_BYTES)
    return ALBIREO_E_SCRATCH;
  void* ws = nullptr;
  int dev = -1;
  albireo_status_t st = scratch_for_current_device(&ws, &dev);
  if (st != ALBIREO_OK) return st;
  {
    // a call whose launches the runtime refused part-way may have left the array non-zero: zero all of
    // it (stream order) before it serves again
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dirty[dev]) {
      const int64_t n = (int64_t)ALBIREO_NOALLOC_SCRATCH_BYTES / 16;
      hipLaunchKernelGGL(k_zero16, dim3(2048), dim3(256), 0, stream, static_cast<uint4*>(ws), n);
      if (hipGetLastError() != hipSuccess) return ALBIREO_E_LAUNCH;
      g_scratch_dirty[dev] = false;
    }
  }
  st = sample_impl(logits, dtype, B, V, ld, nullptr, params, uniforms, nullptr, out_ids, out_logprobs, n_top,
                   out_top_ids, out_top_logprobs, out_flags, ws, (size_t)ALBIREO_NOALLOC_SCRATCH_BYTES, stream);
  if (st == ALBIREO_E_LAUNCH) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    g_scratch_dirty[dev] = true;
  }
  return st;
}

albireo_status_t albireo_sample_step(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                     const albireo_params_t* params, const albireo_step_t* step, int32_t* out_ids,
                                     float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                     float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  if (!step) return ALBIREO_E_INVALID;
  return sample_impl(logits, dtype, B, V, ld, nullptr, params, nullptr, step, out_ids, out_logprobs, n_top,
                     out_top_ids, out_top_logprobs, out_flags, workspace, workspace_bytes, stream);
}

albireo_status_t albireo_sample_sharded(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                        const albireo_shards_t* shards, const albireo_params_t* params,
                                        const float* uniforms, const albireo_step_t* step, int32_t* out_ids,
                                        float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                        float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  if (!shards || (uniforms == nullptr) == (step == nullptr)) return ALBIREO_E_INVALID;
  return sample_impl(logits, dtype, B, V, ld, shards, params, uniforms, step, out_ids, out_logprobs, n_top,
                     out_top_ids, out_top_logprobs, out_flags, workspace, workspace_bytes, stream);
}

albireo_status_t albireo_philox_uniforms(uint64_t seed, uint64_t step, const int64_t* seq_ids, int64_t B,
                                         float* out_uniforms, hipStream_t stream) {
  if (B < 0) return ALBIREO_E_INVALID;
  if (B == 0) return ALBIREO_OK;
  if (!out_uniforms) return ALBIREO_E_INVALID;
  const int64_t blocks = (B + 255) / 256;
  if (blocks > 0x7fffffff) return ALBIREO_E_UNSUPPORTED;
  hipLaunchKernelGGL(k_philox_uniforms, dim3((unsigned)blocks), dim3(256), 0, stream, seed, step, seq_ids, B,
                     out_uniforms);
  return hipGetLastError() == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

albireo_status_t albireo_backfill(const int32_t* ids, const int32_t* dest, int64_t B, int32_t* next_tokens,
                                  int64_t next_len, hipStream_t stream) {
  if (B < 0 || next_len < 0) return ALBIREO_E_INVALID;
  if (B == 0) return ALBIREO_OK;
  if (!ids || !dest || !next_tokens) return ALBIREO_E_INVALID;
  const int64_t blocks = (B + 255) / 256;
  if (blocks > 0x7fffffff) return ALBIREO_E_UNSUPPORTED;
  hipLaunchKernelGGL(k_backfill, dim3((unsigned)blocks), dim3(256), 0, stream, ids, dest, B, next_tokens, next_len);
  return hipGetLastError() == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

albireo_status_t albireo_topk_topp(const float* logits, int64_t B, int64_t V, int64_t ld,
                                   const albireo_params_t* params, float* out_probs, float* out_threshold,
                                   int32_t* out_kept, float* out_log_norm, uint32_t* out_flags,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  albireo_status_t st = check_common(logits, ALBIREO_F32, B, V, ld, nullptr);
  if (st != ALBIREO_OK) return st;
  if (B == 0) return ALBIREO_OK;
  Geometry G;
  if (make_geometry(B, V, ALBIREO_F32, G) != hipSuccess) return ALBIREO_E_LAUNCH;
  if (!G.ok) return ALBIREO_E_UNSUPPORTED;
  st = check_ws(workspace, workspace_bytes, required_ws(G));
  if (st != ALBIREO_OK) return st;
  KArgs a;
  memset(&a, 0, sizeof a);
  a.logits = reinterpret_cast<const unsigned char*>(logits);
  a.B = B;
  a.V = V;
  a.ld = ld;
  a.prm = dev_params(params);
  // the filtered distribution uses temperature and the three filters only
  a.prm.rep = a.prm.freq = a.prm.pres = nullptr;
  a.prm.hist_offsets = nullptr;
  a.prm.hist_ids = nullptr;
  a.prm.hist_len = 0;
  a.out_probs = out_probs;
  a.out_threshold = out_threshold;
  a.out_kept = out_kept;
  a.out_log_norm = out_log_norm;
  a.out_flags = out_flags;
  a.mode = 1;
  a.ws = static_cast<unsigned char*>(workspace);
  return launch_sample(a, G, stream);
}

albireo_status_t albireo_apply_penalties(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V,
                                         int64_t ld, const albireo_params_t* params, float* out_logits,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  (void)workspace;
  (void)workspace_bytes;
  albireo_status_t st = check_common(logits, dtype, B, V, ld, params);
  if (st != ALBIREO_OK) return st;
  if (B == 0) return ALBIREO_OK;
  if (!out_logits) return ALBIREO_E_INVALID;
  // aliasing is only defined for an fp32 input with ld == V (element-wise in place)
  if (static_cast<const void*>(out_logits) == logits && !(dtype == ALBIREO_F32 && ld == V)) return ALBIREO_E_INVALID;
  if (B > 65535) return ALBIREO_E_UNSUPPORTED;
  const DevParams d = dev_params(params);
  PenExtra ex;
  memset(&ex, 0, sizeof ex);
  if (params) {
    ex.prompt_offsets = params->prompt_offsets;
    ex.prompt_ids = params->prompt_ids;
    ex.prompt_len = params->prompt_len;
    if (params->state) {
      ex.st_ids = params->state->ids;
      ex.st_counts = params->state->counts;
      ex.st_len = params->state->len;
      ex.st_cap = params->state->cap;
    }
  }
  const dim3 grid((unsigned)((V + PEN_TILE - 1) / PEN_TILE), (unsigned)B);
  if (dtype == ALBIREO_BF16)
    hipLaunchKernelGGL(k_penalties<BF16T>, grid, dim3(PEN_NT), 0, stream,
                       static_cast<const unsigned char*>(logits), V, ld, d, ex, out_logits);
  else
    hipLaunchKernelGGL(k_penalties<F32T>, grid, dim3(PEN_NT), 0, stream,
                       static_cast<const unsigned char*>(logits), V, ld, d, ex, out_logits);
  return hipGetLastError() == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

const char* albireo_status_string(albireo_status_t s) {
  switch (s) {
    case ALBIREO_OK: return "ok";
    case ALBIREO_E_INVALID: return "invalid argument";
    case ALBIREO_E_UNSUPPORTED: return "unsupported shape";
    case ALBIREO_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case ALBIREO_E_LAUNCH: return "kernel launch failed";
    case ALBIREO_E_SCRATCH: return "shape needs more device scratch than albireo_sample_noalloc holds";
  }
  return "unknown status";
}

}  // extern "C"
