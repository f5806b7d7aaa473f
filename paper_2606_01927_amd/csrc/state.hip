// state.hip -- the per-sequence penalty state: build it from a prompt and output history, and fold each
// step's sampled token into it.
//
// The penalties of the paper's workload (sec. 8.1: repetition, frequency and presence) depend on a
// sequence's prompt and on the tokens it has generated so far.  Sampling from raw histories re-counts
// every id of them at every step; the state instead keeps each sequence's distinct ids with their
// output counts and prompt marks on the device, in ascending id order, and a step adds one token.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "albireo.h"

namespace {

constexpr int INIT_NT = 1024;                          // threads of the build workgroup
constexpr int MAXS = ALBIREO_MAX_STATE_ENTRIES;        // ids a build takes per row
constexpr int IPT = MAXS / INIT_NT;                    // ids per thread in the scans
constexpr uint32_t TAG_PROMPT = 0x80000000u;           // prompt mark of an entry's count
constexpr uint32_t KEY_NONE = ~0u;                     // sorts after every (id, tag) key (V < 2^31 - 16)
constexpr int APP_NT = 256;                            // threads of the append workgroup

// CSR row [lo, hi) of a history, or an empty range and a flag when the offsets are malformed
__device__ __forceinline__ void csr_row(const int64_t* off, int64_t len, int64_t row, int64_t& lo, int64_t& hi,
                                        uint32_t& flags) {
  lo = hi = 0;
  if (!off) return;
  const int64_t a = off[row], b = off[row + 1];
  if (a < 0 || b < a || b > len) {
    flags |= ALBIREO_FLAG_BAD_PARAM;
    return;
  }
  lo = a;
  hi = b;
}

// One workgroup per row: the row's occurrences become keys 2 id + (1 for a prompt occurrence), sorted in
// LDS (ascending id, output occurrences before prompt ones), and every run of one id becomes an entry
// whose count is the number of output occurrences in the run and whose prompt mark is the tag of its
// last key.
__global__ __launch_bounds__(INIT_NT) void k_state_init(albireo_penalty_state_t st, int64_t V, const int64_t* p_off,
                                                        const int32_t* p_ids, int64_t p_len, const int64_t* o_off,
                                                        const int32_t* o_ids, int64_t o_len) {
  __shared__ uint32_t key[MAXS];
  __shared__ uint16_t outs_before[MAXS];  // per entry: output occurrences before its run
  __shared__ uint32_t part[2][INIT_NT / 64];
  __shared__ uint32_t sflags;
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  uint32_t flags = 0;
  int64_t plo, phi, olo, ohi;
  csr_row(p_off, p_len, row, plo, phi, flags);
  csr_row(o_off, o_len, row, olo, ohi, flags);
  const int64_t np = phi - plo, no = ohi - olo;
  int64_t total = np + no;
  if (total > MAXS) {
    flags |= ALBIREO_FLAG_LIMIT;
    total = MAXS;
  }
  const int n = (int)total;
  if (t == 0) sflags = flags;
  __syncthreads();
  uint32_t bad = 0;
  for (int j = t; j < MAXS; j += INIT_NT) {
    uint32_t k = KEY_NONE;
    if (j < n) {
      const bool pr = j < np;
      const int32_t id = pr ? p_ids[plo + j] : o_ids[olo + (j - np)];
      if (id >= 0 && (int64_t)id < V) k = ((uint32_t)id << 1) | (pr ? 1u : 0u);
      else bad = 1;
    }
    key[j] = k;
  }
  if (bad) atomicOr(&sflags, ALBIREO_FLAG_BAD_INPUT);
  int npad = 1;
  while (npad < n) npad <<= 1;
  __syncthreads();
  // bitonic sort of key[0, npad), ascending
  for (int size = 2; size <= npad; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = t; i < (npad >> 1); i += INIT_NT) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const uint32_t x = key[lo], y = key[hi];
        if ((x > y) == up) {
          key[lo] = y;
          key[hi] = x;
        }
      }
      __syncthreads();
    }
  }
  // thread t owns positions [t IPT, t IPT + IPT): inclusive prefixes of run starts and output tags
  int firsts = 0, outs = 0;
  const int j0 = t * IPT;
#pragma unroll
  for (int q = 0; q < IPT; ++q) {
    const int j = j0 + q;
    const uint32_t k = key[j];
    if (k != KEY_NONE) {
      firsts += (j == 0 || (key[j - 1] >> 1) != (k >> 1)) ? 1 : 0;
      outs += (k & 1u) ? 0 : 1;
    }
  }
  // exclusive scans over the threads (two values)
  const int l = t & 63, w = t >> 6;
  int fi = firsts, oi = outs;
  for (int o = 1; o < 64; o <<= 1) {
    const int f2 = __shfl_up(fi, o), o2 = __shfl_up(oi, o);
    if (l >= o) {
      fi += f2;
      oi += o2;
    }
  }
  if (l == 63) {
    part[0][w] = (uint32_t)fi;
    part[1][w] = (uint32_t)oi;
  }
  __syncthreads();
  int fb = fi - firsts, ob = oi - outs, nd = 0;
  for (int q = 0; q < INIT_NT / 64; ++q) {
    if (q < w) {
      fb += (int)part[0][q];
      ob += (int)part[1][q];
    }
    nd += (int)part[0][q];
  }
  const int cap = st.cap;
  int32_t* ids = st.ids + row * cap;
  uint32_t* cnt = st.counts + row * cap;
  // run starts: the entry's id and the output tags before it
  {
    int d = fb - 1, o = ob;
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int j = j0 + q;
      const uint32_t k = key[j];
      if (k != KEY_NONE) {
        if (j == 0 || (key[j - 1] >> 1) != (k >> 1)) {
          ++d;
          outs_before[d] = (uint16_t)o;
          if (d < cap) ids[d] = (int32_t)(k >> 1);
        }
        o += (k & 1u) ? 0 : 1;
      }
    }
  }
  __syncthreads();
  // run ends: the count and the prompt mark
  {
    int d = fb - 1, o = ob;
#pragma unroll
    for (int q = 0; q < IPT; ++q) {
      const int j = j0 + q;
      const uint32_t k = key[j];
      if (k != KEY_NONE) {
        if (j == 0 || (key[j - 1] >> 1) != (k >> 1)) ++d;
        o += (k & 1u) ? 0 : 1;
        const bool last = (j + 1 == MAXS) || (key[j + 1] >> 1) != (k >> 1);
        if (last && d < cap) cnt[d] = (uint32_t)(o - (int)outs_before[d]) | ((k & 1u) ? TAG_PROMPT : 0u);
      }
    }
  }
  if (t == 0) {
    st.len[row] = nd < cap ? nd : cap;
    st.flags[row] = sflags | (nd > cap ? ALBIREO_FLAG_LIMIT : 0u);
  }
}

// One workgroup per row: find the id among the row's entries (they are in ascending order); count one
// more output occurrence, or insert a new entry at its place by moving the larger entries up by one.
__global__ __launch_bounds__(APP_NT) void k_state_append(albireo_penalty_state_t st, int64_t V, const int32_t* tok) {
  __shared__ int s_found, s_below;
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int32_t id = tok[row];
  if (id < 0 || (int64_t)id >= V) return;  // uniform over the workgroup
  const int cap = st.cap;
  int32_t* ids = st.ids + row * cap;
  uint32_t* cnt = st.counts + row * cap;
  const int n = st.len[row];
  if (t == 0) {
    s_found = -1;
    s_below = 0;
  }
  __syncthreads();
  int below = 0;
  for (int e = t; e < n; e += APP_NT) {
    const int32_t v = ids[e];
    if (v == id) s_found = e;
    below += v < id ? 1 : 0;
  }
  if (below) atomicAdd(&s_below, below);
  __syncthreads();
  const int found = s_found, pos = s_below;
  if (found >= 0) {
    if (t == 0) cnt[found] = cnt[found] + 1u;
    return;
  }
  if (n >= cap) {
    if (t == 0) st.flags[row] |= ALBIREO_FLAG_LIMIT;
    return;
  }
  // entries [pos, n) move to [pos + 1, n + 1): all read before any is written
  constexpr int MPT = (ALBIREO_MAX_STATE_ENTRIES + APP_NT - 1) / APP_NT;
  int32_t mi[MPT];
  uint32_t mc[MPT];
#pragma unroll
  for (int q = 0; q < MPT; ++q) {
    const int e = pos + t + q * APP_NT;
    if (e < n) {
      mi[q] = ids[e];
      mc[q] = cnt[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < MPT; ++q) {
    const int e = pos + t + q * APP_NT;
    if (e < n) {
      ids[e + 1] = mi[q];
      cnt[e + 1] = mc[q];
    }
  }
  if (t == 0) {
    ids[pos] = id;
    cnt[pos] = 1u;
    st.len[row] = n + 1;
  }
}

albireo_status_t check_state(const albireo_penalty_state_t* st, int64_t B, int64_t V) {
  if (!st || B < 0 || V <= 0) return ALBIREO_E_INVALID;
  if (V >= ((int64_t)1 << 31) - 16 || B > 0x7fffffff) return ALBIREO_E_UNSUPPORTED;
  if (st->cap < 1 || st->cap > ALBIREO_MAX_STATE_ENTRIES) return ALBIREO_E_INVALID;
  if (B > 0 && (!st->ids || !st->counts || !st->len || !st->flags)) return ALBIREO_E_INVALID;
  return ALBIREO_OK;
}

}  // namespace

extern "C" {

albireo_status_t albireo_penalty_state_init(const albireo_penalty_state_t* state, int64_t B, int64_t V,
                                            const int64_t* prompt_offsets, const int32_t* prompt_ids,
                                            int64_t prompt_len, const int64_t* out_offsets,
                                            const int32_t* out_ids, int64_t out_len, hipStream_t stream) {
  albireo_status_t s = check_state(state, B, V);
  if (s != ALBIREO_OK) return s;
  if (prompt_offsets && (prompt_len < 0 || (prompt_len > 0 && !prompt_ids))) return ALBIREO_E_INVALID;
  if (out_offsets && (out_len < 0 || (out_len > 0 && !out_ids))) return ALBIREO_E_INVALID;
  if (B == 0) return ALBIREO_OK;
  hipLaunchKernelGGL(k_state_init, dim3((unsigned)B), dim3(INIT_NT), 0, stream, *state, V, prompt_offsets, prompt_ids,
                     prompt_len, out_offsets, out_ids, out_len);
  return hipGetLastError() == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

albireo_status_t albireo_penalty_state_append(const albireo_penalty_state_t* state, int64_t B, int64_t V,
                                              const int32_t* ids, hipStream_t stream) {
  albireo_status_t s = check_state(state, B, V);
  if (s != ALBIREO_OK) return s;
  if (B == 0) return ALBIREO_OK;
  if (!ids) return ALBIREO_E_INVALID;
  hipLaunchKernelGGL(k_state_append, dim3((unsigned)B), dim3(APP_NT), 0, stream, *state, V, ids);
  return hipGetLastError() == hipSuccess ? ALBIREO_OK : ALBIREO_E_LAUNCH;
}

}  // extern "C"
