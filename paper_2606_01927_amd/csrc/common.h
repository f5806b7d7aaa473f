// common.h -- device helpers shared by the sampling kernels of this library (one copy per
// translation unit; everything here has internal linkage through the enclosing anonymous namespace).
//
// Included by albireo.hip and stream.hip inside `namespace {`.
#pragma once
constexpr uint32_t SPIN_LIMIT = 1u << 24;
constexpr double FIX_SCALE = 4294967296.0;  // fixed-point scale of the general path's masses
constexpr float MREF0 = -3.0e38f;           // initial sum-exp reference (log2 units)
constexpr float L2E = 1.44269504088896341f;  // fl32(log2 e): exp(z) is evaluated as 2^(z * L2E)

constexpr uint32_t FLAG_GREEDY = ALBIREO_FLAG_GREEDY;
constexpr uint32_t FLAG_EMPTY = ALBIREO_FLAG_EMPTY;
constexpr uint32_t FLAG_BAD_INPUT = ALBIREO_FLAG_BAD_INPUT;
constexpr uint32_t FLAG_BAD_PARAM = ALBIREO_FLAG_BAD_PARAM;
constexpr uint32_t FLAG_LIMIT = ALBIREO_FLAG_LIMIT;
constexpr uint32_t FLAG_TIMEOUT = ALBIREO_FLAG_TIMEOUT;

struct DevParams {
  const float* temperature;
  const int32_t* top_k;
  const float* top_p;
  const float* min_p;
  const float* rep;
  const float* freq;
  const float* pres;
  const int64_t* hist_offsets;
  const int32_t* hist_ids;
  int64_t hist_len;
};


__host__ __device__ constexpr int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// ----------------------------------------------------------------------------------------------
// Scalar helpers
// ----------------------------------------------------------------------------------------------
// order-preserving 32-bit key of a float (larger float -> larger key); -inf maps above 0
__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f);
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);  // negative: ~u, else u | sign bit
}
__device__ __forceinline__ float key2f(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}
// canonical processed logit: fl32(x * r) with -0 -> +0; -inf stays -inf (also when r == 0)
// r is finite and positive (a malformed temperature is replaced), so x r keeps -inf and adding +0
// turns -0 into +0
__device__ __forceinline__ float canon(float x, float r) { return __fadd_rn(__fmul_rn(x, r), 0.0f); }
// penalty overlay of one logit seen c > 0 times in the history
__device__ __forceinline__ float penalise(float x, uint32_t c, float rep, float freq, float pres) {
  float v = (x > 0.0f) ? __fdiv_rn(x, rep) : __fmul_rn(x, rep);
  v = __fsub_rn(v, __fmul_rn(freq, (float)c));
  v = __fsub_rn(v, pres);
  return v;
}
// The penalty overlay of one logit whose history record is cv: bits 0-30 its count in the output, bit 31
// set when it occurs in the prompt.  Repetition covers both; frequency and presence count the output.
__device__ __forceinline__ float penalise_cv(float x, uint32_t cv, float rep, float freq, float pres) {
  const uint32_t c = cv & 0x7fffffffu;
  float v = (x > 0.0f) ? __fdiv_rn(x, rep) : __fmul_rn(x, rep);
  if (c > 0) {
    v = __fsub_rn(v, __fmul_rn(freq, (float)c));
    v = __fsub_rn(v, pres);
  }
  return v;
}

// 2^(a - b) for a <= b; a == b (including both -inf) -> 1
__device__ __forceinline__ float rel2(float a, float b) { return (a == b) ? 1.0f : __builtin_amdgcn_exp2f(a - b); }
// candidate sort key: z descending, then position ascending
__device__ __forceinline__ uint64_t cand_key(float z, int pos) {
  return ((uint64_t)f2key(z) << 32) | (uint32_t)(~(uint32_t)pos);
}
__device__ __forceinline__ float cand_z(uint64_t k) { return key2f((uint32_t)(k >> 32)); }
__device__ __forceinline__ int cand_pos(uint64_t k) { return (int)(~(uint32_t)k); }
__device__ __forceinline__ uint64_t fixmass(float w) { return (uint64_t)((double)w * FIX_SCALE); }

template <class T>
__device__ __forceinline__ T ld_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <class T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }
__device__ __forceinline__ int wave_id() { return (int)(threadIdx.x >> 6); }
__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// ----------------------------------------------------------------------------------------------
// Element types: a 16-byte slot holds 8 bf16 or 4 fp32 logits
// ----------------------------------------------------------------------------------------------
struct BF16T {
  static constexpr int VEC = 8;
  static constexpr int ES = 2;
  static constexpr uint32_t NEG = 0xff80ff80u;  // two bf16 -inf
  __device__ static __forceinline__ float get(const uint4& d, int e) {
    const uint32_t w = (e >> 1) == 0 ? d.x : (e >> 1) == 1 ? d.y : (e >> 1) == 2 ? d.z : d.w;
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  }
  __device__ static __forceinline__ float load1(const unsigned char* row, int64_t i) {
    return __uint_as_float((uint32_t)(reinterpret_cast<const uint16_t*>(row)[i]) << 16);
  }
  // bit e of b selects element e; dword k holds element 2k (low half) and 2k+1 (high half)
  __device__ static __forceinline__ uint4 mask_of(uint32_t b) {
    uint4 m;
    m.x = ((b & 1u) ? 0x0000ffffu : 0u) | ((b & 2u) ? 0xffff0000u : 0u);
    m.y = ((b & 4u) ? 0x0000ffffu : 0u) | ((b & 8u) ? 0xffff0000u : 0u);
    m.z = ((b & 16u) ? 0x0000ffffu : 0u) | ((b & 32u) ? 0xffff0000u : 0u);
    m.w = ((b & 64u) ? 0x0000ffffu : 0u) | ((b & 128u) ? 0xffff0000u : 0u);
    return m;
  }
};
struct F32T {
  static constexpr int VEC = 4;
  static constexpr int ES = 4;
  static constexpr uint32_t NEG = 0xff800000u;
  __device__ static __forceinline__ float get(const uint4& d, int e) {
    const uint32_t w = e == 0 ? d.x : e == 1 ? d.y : e == 2 ? d.z : d.w;
    return __uint_as_float(w);
  }
  __device__ static __forceinline__ float load1(const unsigned char* row, int64_t i) {
    return reinterpret_cast<const float*>(row)[i];
  }
  __device__ static __forceinline__ uint4 mask_of(uint32_t b) {
    uint4 m;
    m.x = (b & 1u) ? ~0u : 0u;
    m.y = (b & 2u) ? ~0u : 0u;
    m.z = (b & 4u) ? ~0u : 0u;
    m.w = (b & 8u) ? ~0u : 0u;
    return m;
  }
};

// ----------------------------------------------------------------------------------------------
// Shared memory of the sampling kernel
// ----------------------------------------------------------------------------------------------
// Compile-time loop: f(std::integral_constant<int, I>) for I = 0 .. N-1 as straight-line code, so a
// register array indexed by I never gets a dynamic index (a rolled loop would put it in scratch).
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(static_cast<F&&>(f), std::make_integer_sequence<int, N>{});
}


// ----------------------------------------------------------------------------------------------
// Wave reductions and scans on DPP: row shifts within the 16-lane rows, then the broadcasts of lanes
// 15 and 31 into the following rows, and a total read from lane 63.  Each step costs a few VALU
// cycles where an LDS permute would cost a round trip.  The combination order is fixed by the lane
// layout, so results are bit-identical from run to run and every lane receives the same total.
// ----------------------------------------------------------------------------------------------
constexpr int DPP_ROW_SHR = 0x110, DPP_WAVE_SHR1 = 0x138, DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;

// v from the lane the control names; lanes without a source (or outside ROWS) get `old`
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xf, false);
}
// inclusive scan in lane order under op, whose identity is id
template <class Op>
__device__ __forceinline__ uint32_t wave_scan_bits(uint32_t v, uint32_t id, Op op) {
  v = op(v, dpp_mov<DPP_ROW_SHR + 1>(id, v));
  v = op(v, dpp_mov<DPP_ROW_SHR + 2>(id, v));
  v = op(v, dpp_mov<DPP_ROW_SHR + 4>(id, v));
  v = op(v, dpp_mov<DPP_ROW_SHR + 8>(id, v));
  v = op(v, dpp_mov<DPP_ROW_BCAST15, 0xa>(id, v));
  v = op(v, dpp_mov<DPP_ROW_BCAST31, 0xc>(id, v));
  return v;
}
// value of lane i (i wave-uniform)
__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int i) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, __builtin_amdgcn_readfirstlane(i));
}
__device__ __forceinline__ int lane_i32(int v, int i) { return (int)lane_u32((uint32_t)v, i); }
__device__ __forceinline__ float lane_f32(float v, int i) { return __uint_as_float(lane_u32(__float_as_uint(v), i)); }
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int i) {
  return ((uint64_t)lane_u32((uint32_t)(v >> 32), i) << 32) | lane_u32((uint32_t)v, i);
}

struct OpFmax {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }
};
struct OpFmin {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const {
    return __float_as_uint(fminf(__uint_as_float(a), __uint_as_float(b)));
  }
};
struct OpFadd {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }
};
struct OpAdd {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; }
};
struct OpOr {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a | b; }
};
struct OpMinU {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return min(a, b); }
};
struct OpMinI {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return (uint32_t)min((int)a, (int)b); }
};
struct OpMaxI {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return (uint32_t)max((int)a, (int)b); }
};

__device__ __forceinline__ float wave_max(float v) {
  return __uint_as_float(lane_u32(wave_scan_bits(__float_as_uint(v), __float_as_uint(-INFINITY), OpFmax{}), 63));
}
__device__ __forceinline__ float wave_min(float v) {
  return __uint_as_float(lane_u32(wave_scan_bits(__float_as_uint(v), __float_as_uint(INFINITY), OpFmin{}), 63));
}
__device__ __forceinline__ float wave_sum(float v) {
  return __uint_as_float(lane_u32(wave_scan_bits(__float_as_uint(v), 0u, OpFadd{}), 63));
}
__device__ __forceinline__ int wave_min_i(int v) {
  return (int)lane_u32(wave_scan_bits((uint32_t)v, 0x7fffffffu, OpMinI{}), 63);
}
__device__ __forceinline__ int wave_max_i(int v) {
  return (int)lane_u32(wave_scan_bits((uint32_t)v, 0x80000000u, OpMaxI{}), 63);
}
__device__ __forceinline__ int wave_sum_i(int v) { return (int)lane_u32(wave_scan_bits((uint32_t)v, 0u, OpAdd{}), 63); }
__device__ __forceinline__ uint32_t wave_or(uint32_t v) { return lane_u32(wave_scan_bits(v, 0u, OpOr{}), 63); }
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  return lane_u32(wave_scan_bits(v, 0xffffffffu, OpMinU{}), 63);
}
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint64_t dpp_mov64(uint64_t v) {
  const uint32_t lo = dpp_mov<CTRL, ROWS>(0u, (uint32_t)v);
  const uint32_t hi = dpp_mov<CTRL, ROWS>(0u, (uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  v += dpp_mov64<DPP_ROW_SHR + 1>(v);
  v += dpp_mov64<DPP_ROW_SHR + 2>(v);
  v += dpp_mov64<DPP_ROW_SHR + 4>(v);
  v += dpp_mov64<DPP_ROW_SHR + 8>(v);
  v += dpp_mov64<DPP_ROW_BCAST15, 0xa>(v);
  v += dpp_mov64<DPP_ROW_BCAST31, 0xc>(v);
  return lane_u64(v, 63);
}
__device__ __forceinline__ int wave_incl_scan_i(int v) { return (int)wave_scan_bits((uint32_t)v, 0u, OpAdd{}); }
__device__ __forceinline__ uint32_t wave_incl_scan_u(uint32_t v) { return wave_scan_bits(v, 0u, OpAdd{}); }
__device__ __forceinline__ float wave_incl_scan(float v) {
  return __uint_as_float(wave_scan_bits(__float_as_uint(v), 0u, OpFadd{}));
}

// Load of a wave-uniform, read-only value through the scalar unit (constant address space): it is
// tracked apart from the vector loads, so waiting for it never waits for row data in flight.
template <class T>
__device__ __forceinline__ T sload(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}


// Values of the per-row parameters whose arrays are NULL (feature off), read in their place so that
// every parameter load is one unconditional scalar load.
__constant__ float kParamDefaults[8] = {1.0f, 1.0f, 0.0f, 1.0f, 0.0f, 0.0f, 0.0f, 0.0f};  // T p min_p rep freq pres u
__constant__ int32_t kZeroI32[2] = {0, 0};
__constant__ int64_t kZeroI64[2] = {0, 0};

// ----------------------------------------------------------------------------------------------
// Counter-based uniforms: Philox-4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC 2011).  Each
// round forms the 64-bit products of counter words 0 and 2 with two fixed odd multipliers, and the
// new counter is (high half of the second product ^ word 1 ^ key 0, its low half, high half of the
// first product ^ word 3 ^ key 1, its low half); the key advances by two Weyl constants per round.
// A row's uniform: counter (step, sequence id) as four 32-bit words (low word first), key = seed, and
// the top 24 bits of the first output word scaled by 2^-24, so u lies in [0, 1) on a 2^-24 grid.
// Every argument here is wave-uniform, so the rounds run on the scalar unit.
// ----------------------------------------------------------------------------------------------
__host__ __device__ __forceinline__ float philox_uniform(uint64_t seed, uint64_t step, uint64_t seq) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t c0 = (uint32_t)step, c1 = (uint32_t)(step >> 32), c2 = (uint32_t)seq, c3 = (uint32_t)(seq >> 32);
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t a0 = (uint64_t)M0 * c0, a1 = (uint64_t)M1 * c2;
    const uint32_t n0 = (uint32_t)(a1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(a0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)a1;
    c3 = (uint32_t)a0;
    c0 = n0;
    c2 = n2;
    k0 += W0;
    k1 += W1;
  }
  return (float)(c0 >> 8) * (1.0f / 16777216.0f);
}
