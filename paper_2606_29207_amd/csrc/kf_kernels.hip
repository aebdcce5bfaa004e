// gfx950 kernels of the weightless attention node's decode step
// (KernelFlume, arXiv 2606.29207, Section 3.2 steps 3-4, Section 5.1):
//   append_kernel   -- tail append of the step's K/V token
//   partial_kernel  -- local attention over token-range routes -> (o, lse)
//   order_kernel    -- dispatch order of a split launch of several rounds
//   combine_kernel  -- in-range reduction of a split unit's ranges
//   merge_kernel    -- log-sum-exp merge of the partials of each sequence
//
// partial_kernel is HBM-bound (4 flop per KV byte at 4 query heads per KV
// head).  Four waves own a (route, KV head) unit -- or, when the host plans
// chunks, one of its ceil(pages / chunk_pages) page ranges: a 256-thread
// workgroup, two per CU, or one half of a 512-thread workgroup that holds
// two short unsplit bf16 units, one per CU.  Wave w takes tiles w, w+4, ... of
// the range, its full tiles taken from a per-route starting offset, so the
// summation order is fixed and results are bitwise reproducible (and the
// same for any placement of the pages).  Each wave streams tiles of 2 (bf16)
// or 4 (fp8) pages:
//   * lane (grp = lane/16, i = lane%16).  For q.K^T the MFMA A operand row i
//     is token (page i/4 of the tile, slot 4c + i%4) for c = 0..3, so the
//     16x16 result lands with lane (grp, head i) holding all 16 scores of
//     page grp of the tile.  Those are exactly the P^T values the same lane
//     feeds as the B operand of p.V, whose A operand is read straight from
//     the dimension-major V page (V^T rows are contiguous in slots): no LDS
//     or cross-lane traffic between the two products.
//   * both products use v_mfma_f32_16x16x32_bf16; query heads of the group
//     fill the N = 16 columns (G <= 16, the rest zero).
//   * p (fp32) enters p.V as bf16 hi + bf16 lo, two MFMAs, so the products
//     carry ~2^-17 relative error instead of bf16's 2^-9.
//   * all 32 loads of a tile are issued before any of its arithmetic, and
//     the page ids of the wave's next tile are fetched a tile ahead.
//   * softmax state per head is shared by the four lane groups (max reduced
//     across groups per tile), the running sum is kept per lane and reduced
//     once at the end; the four waves are combined through LDS.
// Workgroups never exchange data with each other inside a kernel: when a
// unit is chunked, the chunk partials go to the workspace and combine_kernel
// (the next launch on the stream) merges them in chunk order, so results are
// deterministic.
#include <atomic>
#include <mutex>
#include <type_traits>

#include "kf_internal.h"


namespace kf {
namespace {

// Slice index of (page, KV head) in a pool: page-major pools are
// [num_pages][Hkv][...], head-major ones [Hkv][num_pages][...].
__device__ __forceinline__ size_t pool_slice(int page, int g, int H, int P, int32_t head_major) {
  return head_major ? (size_t)g * P + page : (size_t)page * H + g;
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kThreads = kWaves * 64;
constexpr int kLdsStride = kDim + 4;  // padded row of the per-wave output buffer


__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }
__device__ __forceinline__ float qnan() { return __builtin_nanf(""); }

__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// 16 E4M3FN codes (one dword = 4 codes, lowest byte first) -> 16 bf16 in two
// 8-element operands, exactly (every E4M3 value is a bf16 value).
__device__ __forceinline__ void fp8x16_to_bf16(u32x4 codes, u32x4& lo8, u32x4& hi8) {
  uint32_t o[8];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    o[2 * w] = __builtin_bit_cast(uint32_t,
                                  __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes[w], 1.0f, false));
    o[2 * w + 1] = __builtin_bit_cast(uint32_t,
                                      __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes[w], 1.0f, true));
  }
  lo8 = u32x4{o[0], o[1], o[2], o[3]};
  hi8 = u32x4{o[4], o[5], o[6], o[7]};
}

template <class T>
__device__ __forceinline__ u32x4 ld16(const T* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// K/V pages are read exactly once per step: stream them with the
// non-temporal hint so they do not displace reusable lines in the caches.
template <class T>
__device__ __forceinline__ u32x4 ld16_stream(const T* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// ------------------------------------------------------------------- append
// float32 -> E4M3FN code, round to nearest even, clamped to +-448 (finite
// input); the sign bit is the input's.  Normal range: the 3 leading mantissa
// bits rounded at bit 20 (a carry moves into the exponent); below 2^-6 the
// grid is uniform with step 2^-9.
__device__ __forceinline__ uint32_t e4m3_rne(float v) {
  const uint32_t sign = (__builtin_bit_cast(uint32_t, v) >> 24) & 0x80u;
  const float a = fminf(fabsf(v), 448.0f);
  uint32_t code;
  if (a < 0.015625f) {
    code = (uint32_t)__builtin_rintf(a * 512.0f);
  } else {
    const uint32_t ab = __builtin_bit_cast(uint32_t, a);
    const uint32_t man = ab & 0x7FFFFFu;
    const uint32_t rounded = man + 0x7FFFFu + ((man >> 20) & 1u);
    code = ((((ab >> 23) & 0xFFu) - 120u) << 3) + (rounded >> 20);
  }
  return sign | code;
}

// E4M3FN code -> float32 (exact; the code widens to bf16, then to fp32).
__device__ __forceinline__ float e4m3_value(uint32_t code) {
  const uint32_t b2 = __builtin_bit_cast(uint32_t,
                                         __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(code, 1.0f, false));
  return __builtin_bit_cast(float, b2 << 16);
}

// The E4M3 append rule for one token of one (page, KV head) of K (is_v
// false, page [slot][d]) or V (page [d][slot]), by one wave whose lane holds
// dims 2 lane, 2 lane + 1; all arithmetic in float32.  The first token of a
// page sets scale = amax/28 (16x headroom below 448); a later token with
// amax > 448*scale first re-encodes the page's earlier slots to amax/28; the
// token is stored as RNE(x/scale).  Returns the page's scale afterwards
// (old_scale is ignored for slot 0); the caller stores it.
__device__ float append_e4m3_head(uint8_t* page, float old_scale, int slot, bool is_v,
                                  const uint16_t* x_bits, int lane) {
  const int d0 = 2 * lane;
  const float x0 = __builtin_bit_cast(float, (uint32_t)x_bits[d0] << 16);
  const float x1 = __builtin_bit_cast(float, (uint32_t)x_bits[d0 + 1] << 16);
  float amax = fmaxf(fabsf(x0), fabsf(x1));
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m));
  auto at = [&](int s_, int d_) -> uint8_t* {
    return page + (is_v ? d_ * kPage + s_ : s_ * kDim + d_);
  };
  float scale;
  if (slot == 0) {
    scale = amax > 0.0f ? amax / 28.0f : 1.0f;
  } else {
    scale = old_scale;
    if (amax > 448.0f * scale) {
      const float fresh = amax / 28.0f;
      for (int s_ = 0; s_ < slot; ++s_) {
        uint8_t* p0 = at(s_, d0);
        uint8_t* p1 = at(s_, d0 + 1);
        const float v0 = e4m3_value(*p0) * scale;
        const float v1 = e4m3_value(*p1) * scale;
        *p0 = (uint8_t)e4m3_rne(v0 / fresh);
        *p1 = (uint8_t)e4m3_rne(v1 / fresh);
      }
      scale = fresh;
    }
  }
  *at(slot, d0) = (uint8_t)e4m3_rne(x0 / scale);
  *at(slot, d0 + 1) = (uint8_t)e4m3_rne(x1 / scale);
  return scale;
}

template <bool FP8>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  const int b = blockIdx.x;
  const int r = a.tail_route[b];
  if (r < 0) return;
  int flag = 0;
  int32_t seq = 0, tb = 0, te = 0, base = 0, cap = 0, pid = 0;
  if (r >= a.num_routes) {
    flag = KF_EFLAG_BAD_ROUTE;
  } else {
    const int32_t* rp = reinterpret_cast<const int32_t*>(a.routes + r);
    seq = rp[0]; tb = rp[2]; te = rp[3]; base = rp[4]; cap = rp[5];
    const int j = te - tb;
    if (seq != b || j < 0) {
      flag = KF_EFLAG_BAD_ROUTE;
    } else if (j / kPage >= cap) {
      flag = KF_EFLAG_TAIL_FULL;
    } else if (base < 0 || (int64_t)base + j / kPage >= a.num_page_ids) {
      flag = KF_EFLAG_BAD_ROUTE;
    } else {
      pid = a.page_ids[base + j / kPage];
      if (pid < 0 || pid >= a.num_pages) flag = KF_EFLAG_BAD_PAGE;
    }
  }
  if (flag) {
    if (threadIdx.x == 0) atomicOr(a.err_flags, flag);
    return;
  }
  const int slot = (te - tb) % kPage;
  const int H = a.num_kv_heads;
  if constexpr (!FP8) {
    uint16_t* kp = static_cast<uint16_t*>(a.k_pool);
    uint16_t* vp = static_cast<uint16_t*>(a.v_pool);
    for (int e = threadIdx.x; e < H * kDim; e += blockDim.x) {
      const int g = e / kDim, d = e % kDim;
      const size_t head = pool_slice(pid, g, H, a.num_pages, a.head_major);
      const uint16_t kv = a.k_new[((size_t)b * H + g) * kDim + d];
      const uint16_t vv = a.v_new[((size_t)b * H + g) * kDim + d];
      kp[(head * kPage + slot) * kDim + d] = kv;
      vp[(head * kDim + d) * kPage + slot] = vv;
    }
  } else {
    // One wave per (KV head, K|V)
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (int pr = w; pr < 2 * H; pr += nw) {
      const int g = pr >> 1;
      const bool is_v = pr & 1;
      float* scale = (is_v ? a.v_scale : a.k_scale) + (size_t)pid * H + g;
      uint8_t* page = static_cast<uint8_t*>(is_v ? a.v_pool : a.k_pool) +
                      pool_slice(pid, g, H, a.num_pages, a.head_major) * (kPage * kDim);
      const float s_new = append_e4m3_head(page, *scale, slot, is_v,
                                           (is_v ? a.v_new : a.k_new) + ((size_t)b * H + g) * kDim,
                                           lane);
      if (lane == 0) *scale = s_new;
    }
  }
  __syncthreads();  // every thread has read tok_end before it moves
  if (threadIdx.x == 0) a.routes[r].tok_end = te + 1;
}

// ------------------------------------------------------------------ partial
// The murmur3 32-bit finaliser: a route's tile walk starts at
// route_hash(route) / 2^32 of its full tiles.
__device__ __forceinline__ uint32_t route_hash(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85EBCA6Bu;
  x ^= x >> 13;
  x *= 0xC2B2AE35u;
  x ^= x >> 16;
  return x;
}

struct RouteView {
  int seq, n, npages, base;
  bool bad;
  bool app;       // fused step: this route takes the step's token (local index n - 1)
  int app_pid;    // page id and slot that receive it
  int app_slot;
};

// The append rule of append_kernel, seen from the route: route r takes the
// step's token iff it is its sequence's tail and the token's page is
// reserved, listed and inside the pool.  The merge kernel takes the same
// decision from the sequence side (tail_append_status).
__device__ __forceinline__ bool fused_append(const PartialArgs& a, int r, int seq, int j, int base,
                                             int cap, int& pid) {
  if (!a.tail_route || seq < 0 || seq >= a.num_seqs || a.tail_route[seq] != r) return false;
  if (j < 0 || j / kPage >= cap || base < 0 || (int64_t)base + j / kPage >= a.num_page_ids)
    return false;
  pid = a.page_ids[base + j / kPage];
  return pid >= 0 && pid < a.num_pages;
}

// Route row r as the kernels see it, with the device-side consistency checks
// (in a fused step, after the step's append).
__device__ __forceinline__ RouteView read_route(const PartialArgs& a, int r) {
  const int32_t* rp = reinterpret_cast<const int32_t*>(a.routes + r);
  RouteView v;
  v.seq = rp[0];
  const int tb = rp[2], te = rp[3], cap = rp[5];
  v.base = rp[4];
  v.n = te - tb;
  v.app_pid = 0;
  v.app = fused_append(a, r, v.seq, v.n, v.base, cap, v.app_pid);
  v.app_slot = v.n & (kPage - 1);
  if (v.app) v.n += 1;
  v.npages = v.n > 0 ? (v.n + kPage - 1) / kPage : 0;
  v.bad = v.seq < 0 || v.seq >= a.num_seqs || v.n < 0 || v.base < 0 || v.npages > cap ||
          v.npages > a.max_pages_per_route || (int64_t)v.base + v.npages > a.num_page_ids;
  return v;
}

// Fused step: write the step's token of KV head g into the route's page
// (publish_to_workgroup then makes it visible to every wave of the
// workgroup before any of them loads the page).  fp8 pools follow the E4M3
// append rule (waves 0 and 1 take K and V) and hand the page's new scales to
// the workgroup in s_app[0..1]: the scalar cache is not coherent with vector
// stores, so the tail page's scales must not be read back through scalar
// loads in this launch.  tid: thread index within the unit's 256 threads.
template <bool FP8>
__device__ __forceinline__ void store_new_token(const PartialArgs& a, const RouteView& rv, int g,
                                                int tid, float* s_app) {
  const int H = a.num_kv_heads;
  const uint16_t* kn = a.k_new + ((size_t)rv.seq * H + g) * kDim;
  const uint16_t* vn = a.v_new + ((size_t)rv.seq * H + g) * kDim;
  const size_t head = pool_slice(rv.app_pid, g, H, a.num_pages, a.head_major);
  if constexpr (!FP8) {
    if (tid < kDim) {
      static_cast<uint16_t*>(a.k_pool_w)[(head * kPage + rv.app_slot) * kDim + tid] = kn[tid];
      static_cast<uint16_t*>(a.v_pool_w)[(head * kDim + tid) * kPage + rv.app_slot] = vn[tid];
    }
  } else {
    const int wv = tid >> 6, lane = tid & 63;
    if (wv < 2) {
      const bool is_v = wv == 1;
      // scales are [num_pages][Hkv] in either pool layout
      float* scale = (is_v ? a.v_scale_w : a.k_scale_w) + (size_t)rv.app_pid * H + g;
      uint8_t* page = static_cast<uint8_t*>(is_v ? a.v_pool_w : a.k_pool_w) + head * (kPage * kDim);
      const float s_new = append_e4m3_head(page, *scale, rv.app_slot, is_v, is_v ? vn : kn, lane);
      if (lane == 0) {
        *scale = s_new;
        s_app[wv] = s_new;
      }
    }
  }
}

// Orders the workgroup's earlier global stores before every later load of
// its waves (the waves of a workgroup share the compute unit's L1).
__device__ __forceinline__ void publish_to_workgroup() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Tile geometry.  A wave tile is TP pages: 2 for bf16 (16 KiB of K+V), 4 for
// fp8 (also 16 KiB).  Lane (grp = lane/16, li = lane%16):
//   q.K^T MFMA c (c < TP) takes K row li = token (kpage(li), kslot(c, li));
//   the 16x16 result gives lane (grp, head li) the TP*4 slots
//   vslot0 + 4c + r4 of tile page vpage(grp), which are exactly the k-slots
//   the lane feeds to p.V (NH = TP/2 MFMAs of 8 slots per 16-dim block).
template <bool FP8>
struct Geo {
  static constexpr int TP = FP8 ? 4 : 2;  // pages per tile
  static constexpr int NC = TP;           // q.K^T MFMAs of 16 rows per tile
  static constexpr int NH = TP / 2;       // p.V MFMAs (8 slots each) per 16-dim block
  static __device__ __forceinline__ int kpage(int li) { return FP8 ? li >> 2 : li >> 3; }
  static __device__ __forceinline__ int kslot0(int li) {
    return FP8 ? (li & 3) : 8 * ((li >> 2) & 1) + (li & 3);
  }
  static __device__ __forceinline__ int vpage(int grp) { return FP8 ? grp : grp >> 1; }
  static __device__ __forceinline__ int vslot0(int grp) { return FP8 ? 0 : 8 * (grp & 1); }
};

// Raw bytes of one tile as one lane loads them.
template <bool FP8>
struct TileRaw;
template <>
struct TileRaw<false> {
  u32x4 k[2][4];  // [c][kk]: 8 bf16 of K row kslot(c), dims 32*kk + 8*grp ..
  u32x4 v[8];     // [b8]: 8 bf16 of V^T row d = 16*b8 + li, slots vslot0 ..
};
template <>
struct TileRaw<true> {
  u32x4 k[4][2];  // [c][pp]: 16 E4M3 of K row kslot(c), dims 64*pp + 16*grp ..
  u32x4 v[8];     // [b8]: the 16 E4M3 slots of V^T row d = 16*b8 + li
  float ks, vs;   // K and V scales of the lane's page (vpage)
};

// Wave-uniform description of one tile: its first route-local page and the
// page ids of its (up to four) pages.
struct TileInfo {
  int tp0;
  int pid0, pid1, pid2, pid3;
};

template <class T>
__device__ __forceinline__ T pick4(T v0, T v1, T v2, T v3, int i) {
  return (i & 2) ? ((i & 1) ? v3 : v2) : ((i & 1) ? v1 : v0);
}

// UPW = units per workgroup.  1: a 256-thread workgroup owns one (route, KV
// head) unit or one chunk of it, two workgroups per CU.  2 (unsplit bf16
// launches of units of at most kMaxPagesTwoUnit pages): a 512-thread
// workgroup owns units u and u + gridDim.z, waves 0-3 the first and 4-7 the
// second, one workgroup per CU, so both units of a CU start at once.  In
// that mode all 512 threads reach every barrier: a half without work (no
// unit, a bad or empty one) skips its work, never the barriers.
template <bool FP8, int UPW, bool HM>
__global__ __launch_bounds__(kThreads * UPW, 2 / UPW) void partial_kernel(PartialArgs a) {
  using GeoT = Geo<FP8>;
  constexpr int TP = GeoT::TP, NC = GeoT::NC, NH = GeoT::NH;
  __shared__ float s_o_u[UPW][kWaves][KF_MAX_GROUP][kLdsStride];
  __shared__ float s_m_u[UPW][kWaves][KF_MAX_GROUP];
  __shared__ float s_l_u[UPW][kWaves][KF_MAX_GROUP];
  __shared__ float s_fm_u[UPW][KF_MAX_GROUP];
  __shared__ float s_fl_u[UPW][KF_MAX_GROUP];
  __shared__ float s_app_u[UPW][2];  // fused fp8 append: the tail page's new K and V scales
  // Each wave's half is uniform, but taking it into a scalar register
  // (readfirstlane) made the compiler keep the main loop's next tile in
  // flight for less of each iteration: 2% slower on the Llama layer.
  const int half = UPW == 2 ? (int)(threadIdx.x / kThreads) : 0;
  auto& s_o = s_o_u[half];
  auto& s_m = s_m_u[half];
  auto& s_l = s_l_u[half];
  auto& s_fm = s_fm_u[half];
  auto& s_fl = s_fl_u[half];
  float* s_app = s_app_u[half];

  int c = blockIdx.x;
  int g = blockIdx.y, u = blockIdx.z + half * gridDim.z;  // u: position in the launch
  if (UPW == 1 && a.order) {
    // a split launch of several rounds: take the work item of this
    // workgroup's place in the dispatch order; places past the last item
    // have no work
    const uint32_t i = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    if (i >= a.order[0]) return;
    const uint32_t e0 = a.order[2 + 2 * (size_t)i], e1 = a.order[3 + 2 * (size_t)i];
    u = (int)e0;
    g = (int)(e1 >> 16);
    c = (int)(e1 & 0xFFFFu);
  }
  if constexpr (FP8) {
    // Unsplit fp8 units: workgroups are dealt round-robin over the 8 XCDs.
    // Give XCD k the k-th eighth of the (head, route) space instead, so the
    // heads of a route, whose per-page scales share cache lines, meet in one
    // L2 (the fp8 layer reads ~1% faster; bf16 pools gain nothing from it).
    const unsigned NT = gridDim.y * gridDim.z;
    if (gridDim.x == 1 && (NT & 7u) == 0) {
      const unsigned L = blockIdx.y + gridDim.y * blockIdx.z;
      const unsigned Lp = (L & 7u) * (NT >> 3) + (L >> 3);
      g = Lp % gridDim.y;
      u = Lp / gridDim.y;
    }
  }
  const int G = a.group, Hq = a.num_q_heads, H = a.num_kv_heads;
  const int tid = threadIdx.x & (kThreads - 1), lane = tid & 63, grp = lane >> 4, li = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hq0 = g * G;

  // ---- this unit's page range [p0, p1), or no work for this half: outputs
  // of a bad or empty route are written here
  bool work = false, writer = false;
  int r = -1, nchunks = 1, p0 = 0, p1 = 0;
  RouteView rv{};
  if (u < a.num_units_routes) {
    r = a.route_list ? a.route_list[u] : u;
    if (r < 0 || r >= a.num_routes) {  // a list entry naming no route: nothing to write
      if (c == 0 && g == 0 && tid == 0) atomicOr(a.err_flags, KF_EFLAG_BAD_ROUTE);
    } else {
      rv = read_route(a, r);
      if (rv.bad || rv.npages == 0) {
        if (c == 0) {
          if (rv.app) store_new_token<FP8>(a, rv, g, tid, s_app);  // the pool takes the token all the same
          const float ov = rv.bad ? qnan() : 0.0f, lv = rv.bad ? qnan() : neg_inf();
          for (int e = tid; e < G * kDim; e += kThreads)
            a.o_part[((size_t)r * Hq + hq0 + e / kDim) * kDim + e % kDim] = ov;
          if (tid < G) a.lse_part[(size_t)r * Hq + hq0 + tid] = lv;
          if (rv.bad && tid == 0) atomicOr(a.err_flags, KF_EFLAG_BAD_ROUTE);
        }
      } else {
        nchunks = (rv.npages + a.chunk_pages - 1) / a.chunk_pages;
        if (c < nchunks) {
          work = true;
          writer = rv.app && c == nchunks - 1;  // the chunk with the last page
          p0 = (int)((int64_t)c * rv.npages / nchunks);
          p1 = (int)((int64_t)(c + 1) * rv.npages / nchunks);
        }
      }
    }
  }
  if (writer) store_new_token<FP8>(a, rv, g, tid, s_app);
  if constexpr (UPW == 1) {
    if (!work) return;
    if (writer) publish_to_workgroup();
  } else {
    publish_to_workgroup();
  }
  const int seq = rv.seq, n = rv.n;
  const int app_page = (rv.n - 1) >> 4;             // route-local page of the new token
  const int ntiles = (p1 - p0 + TP - 1) / TP;
  const int lim = min(n, p1 * kPage);  // route-local token bound of this range
  const int32_t* __restrict__ pids = a.page_ids + rv.base;
  // All workgroups start together and stream at about the same pace, so
  // without care every route reads the same offset of its range at the same
  // moment, and in a contiguous pool (routes of a sequence equal sizes apart)
  // the DRAM channels hit at each moment then depend on the pool's layout:
  // the same work ran up to ~9% slower on some page reservations.  Each route
  // therefore walks its full tiles starting from its own offset, rot, taken
  // from a hash of the route index (the murmur3 finaliser), the same for
  // every KV head and chunk of the route, so the heads keep reading the same
  // pages together.  A hash and not a low-discrepancy sequence: offsets
  // spread evenly by the golden ratio made layers with 2 and 16 KV heads
  // stream 8-10% slower (the evenly spaced offsets of equally sized routes
  // meet the same DRAM channels), and per-head offsets lost 1-2% on 4 and 8
  // heads.  A partial last tile keeps its place at the end and is computed
  // masked.  The order depends on the route index only, never on page ids.
  const int nfull = (lim == p1 * kPage && (p1 - p0) % TP == 0) ? ntiles : ntiles - 1;
  const int rot =
      nfull > 1 ? (int)(((uint64_t)route_hash((uint32_t)r) * (uint32_t)nfull) >> 32) : 0;

  auto next_tile = [&](int cur) -> int { return cur + kWaves; };  // wave w: w, w+4, ...

  // Page ids are uniform, so they arrive through scalar loads; a page past
  // the range or outside the pool reads page 0 and is masked (its p set to 0
  // whatever its scales hold) or flagged.  fp8 page scales arrive with the
  // tile's vector loads instead, each lane loading those of its own page: a
  // scalar load of a scale would wait on the scalar load of its page id, and
  // every wait on a scalar load waits on all of them (fp8 layer 1.9% faster).
  bool pid_bad = false;
  auto page_at = [&](int pg) -> int {  // page id of route-local page pg of the range
    const bool in = pg < p1;
    int v = pids[in ? pg : p0];
    v = in ? v : 0;
    if (v < 0 || v >= a.num_pages) {
      pid_bad = true;
      v = 0;
    }
    return v;
  };
  auto tile_info = [&](int tile) -> TileInfo {  // tile: index within the range
    TileInfo t;
    const int tr = tile < nfull ? (tile + rot < nfull ? tile + rot : tile + rot - nfull) : tile;
    t.tp0 = p0 + tr * TP;
    t.pid0 = page_at(t.tp0);
    t.pid1 = page_at(t.tp0 + 1);
    t.pid2 = TP > 2 ? page_at(t.tp0 + 2) : 0;
    t.pid3 = TP > 2 ? page_at(t.tp0 + 3) : 0;
    return t;
  };

  const int kpage = GeoT::kpage(li), vpage = GeoT::vpage(grp);
  const size_t head_elems = (size_t)kPage * kDim;  // elements of one (page, kv head)
  const int koff = GeoT::kslot0(li) * kDim + (FP8 ? 16 : 8) * grp;
  const int voff = li * kPage + GeoT::vslot0(grp);

  auto issue = [&](TileRaw<FP8>& t, const TileInfo& ti) {
    const int pk = pick4(ti.pid0, ti.pid1, ti.pid2, ti.pid3, kpage);
    const int pv = pick4(ti.pid0, ti.pid1, ti.pid2, ti.pid3, vpage);
    const size_t hk = (HM ? (size_t)g * a.num_pages + pk : (size_t)pk * H + g) * head_elems;
    const size_t hv = (HM ? (size_t)g * a.num_pages + pv : (size_t)pv * H + g) * head_elems;
    if constexpr (!FP8) {
      const uint16_t* kb = static_cast<const uint16_t*>(a.k_pool) + hk + koff;
      const uint16_t* vb = static_cast<const uint16_t*>(a.v_pool) + hv + voff;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) t.k[cc][kk] = ld16_stream(kb + cc * 4 * kDim + 32 * kk);
#pragma unroll
      for (int b8 = 0; b8 < 8; ++b8) t.v[b8] = ld16_stream(vb + b8 * 16 * kPage);
    } else {
      const uint8_t* kb = static_cast<const uint8_t*>(a.k_pool) + hk + koff;
      const uint8_t* vb = static_cast<const uint8_t*>(a.v_pool) + hv + voff;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) t.k[cc][pp] = ld16_stream(kb + cc * 4 * kDim + 64 * pp);
#pragma unroll
      for (int b8 = 0; b8 < 8; ++b8) t.v[b8] = ld16_stream(vb + b8 * 16 * kPage);
      t.ks = a.k_scale[(size_t)pv * H + g];
      t.vs = a.v_scale[(size_t)pv * H + g];
    }
  };

  // B operand of q.K^T: query head hq0 + li (zero columns past the group).
  u32x4 qb[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int d0 = FP8 ? 64 * (kk >> 1) + 16 * grp + 8 * (kk & 1) : 32 * kk + 8 * grp;
    qb[kk] = work && li < G ? ld16(a.q + ((size_t)seq * Hq + hq0 + li) * kDim + d0)
                           : u32x4{0, 0, 0, 0};
  }

  f32x4 oacc[8];
#pragma unroll
  for (int b8 = 0; b8 < 8; ++b8) oacc[b8] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = neg_inf(), l_run = 0.0f;

  // MASK: V bits of slots past the range are zeroed (all ones for a full
  // tile).  Only a wave's final tile can hold such slots, so masking is a
  // compile-time property and the steady-state loop has no branch.
  auto compute = [&](const TileRaw<FP8>& t, const TileInfo& ti, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    // ---- S^T = K Q^T (fp8 codes widen to bf16 right before their MFMA)
    f32x4 s[NC];
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      s[cc] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (!FP8) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) s[cc] = mfma16(t.k[cc][kk], qb[kk], s[cc]);
      } else {
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          u32x4 k0, k1;
          fp8x16_to_bf16(t.k[cc][pp], k0, k1);
          s[cc] = mfma16(k0, qb[2 * pp], s[cc]);
          s[cc] = mfma16(k1, qb[2 * pp + 1], s[cc]);
        }
      }
    }
    float ks = a.scale_log2, vs = 1.0f;
    if constexpr (FP8) {
      float kss = t.ks;
      vs = t.vs;
      if (writer && ti.tp0 + vpage == app_page) {  // the tail page's scales were just written
        kss = s_app[0];
        vs = s_app[1];
      }
      ks *= kss;
    }
    const int tok0 = (ti.tp0 + vpage) * kPage + GeoT::vslot0(grp);  // route-local token, c = r4 = 0
    float mt = neg_inf();
#pragma unroll
    for (int cc = 0; cc < NC; ++cc)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const float v = (tok0 + 4 * cc + r4 < lim) ? s[cc][r4] * ks : neg_inf();
        s[cc][r4] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2_fast(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int b8 = 0; b8 < 8; ++b8) oacc[b8] *= alpha;

    // ---- P^T operands: half h2 holds slots 8*h2 + j (j < 8) of the lane's
    // range, i.e. MFMA c = 2*h2 + j/4, row r4 = j%4; bf16 hi + lo
    u32x4 phi[NH], plo[NH];
#pragma unroll
    for (int h2 = 0; h2 < NH; ++h2)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int cc = 2 * h2 + (jj >> 1), r4 = 2 * (jj & 1);
        const float e0 = exp2_fast(s[cc][r4] - m_new);
        const float e1 = exp2_fast(s[cc][r4 + 1] - m_new);
        l_run += e0 + e1;
        float x0 = e0 * vs, x1 = e1 * vs;
        if constexpr (MASK && FP8) {  // a masked slot adds nothing, whatever its page's scales
          const int t0 = tok0 + 8 * h2 + 2 * jj;
          x0 = t0 < lim ? x0 : 0.0f;
          x1 = t0 + 1 < lim ? x1 : 0.0f;
        }
        const uint32_t b0 = __builtin_bit_cast(uint32_t, x0) & 0xFFFF0000u;
        const uint32_t b1 = __builtin_bit_cast(uint32_t, x1) & 0xFFFF0000u;
        phi[h2][jj] = (b0 >> 16) | b1;
        plo[h2][jj] = pack_bf16_rne(x0 - __builtin_bit_cast(float, b0),
                                    x1 - __builtin_bit_cast(float, b1));
      }

    // ---- O^T += V^T P^T; V of slots past the range is zeroed (unused slots
    // may hold anything)
    uint32_t msk[NH][4];
#pragma unroll
    for (int h2 = 0; h2 < NH; ++h2)
#pragma unroll
      for (int wd = 0; wd < 4; ++wd) {
        const int t0 = tok0 + 8 * h2 + 2 * wd;
        msk[h2][wd] = (t0 < lim ? 0x0000FFFFu : 0u) | (t0 + 1 < lim ? 0xFFFF0000u : 0u);
      }
#pragma unroll
    for (int b8 = 0; b8 < 8; ++b8) {
      u32x4 vr[NH];
      if constexpr (!FP8) vr[0] = t.v[b8];
      else fp8x16_to_bf16(t.v[b8], vr[0], vr[1]);
      if constexpr (MASK) {
#pragma unroll
        for (int h2 = 0; h2 < NH; ++h2)
#pragma unroll
          for (int wd = 0; wd < 4; ++wd) vr[h2][wd] &= msk[h2][wd];
      }
#pragma unroll
      for (int h2 = 0; h2 < NH; ++h2) {
        oacc[b8] = mfma16(vr[h2], phi[h2], oacc[b8]);
        oacc[b8] = mfma16(vr[h2], plo[h2], oacc[b8]);
      }
    }
  };

  // ---- two register buffers: while one tile is computed, the loads of the
  // wave's next tile are in flight.  Between issuing a tile and computing
  // the previous one there is no branch, so the compiler waits only for the
  // tile it computes; tile ids and their page ids are fetched a tile ahead.
  // A wave's tile ids increase, so a tile computed inside the loop always
  // precedes one already issued and is full; only the tile computed after
  // the loop can be the range's last and is computed masked.
  TileRaw<FP8> ra, rb;
  const std::integral_constant<bool, false> full{};
  const std::integral_constant<bool, true> masked{};
  if (w < ntiles) {
    const int last = ntiles - 1;
    TileInfo ia = tile_info(w);
    issue(ra, ia);
    int tb = next_tile(w);
    TileInfo ib = tile_info(min(tb, last));
    bool final_in_b = false;
    while (true) {
      if (tb > last) break;
      issue(rb, ib);
      const int tn = next_tile(tb);
      const TileInfo in = tile_info(min(tn, last));
      __builtin_amdgcn_sched_barrier(0);
      compute(ra, ia, full);
      if (tn > last) {
        final_in_b = true;
        break;
      }
      ia = in;
      issue(ra, ia);
      tb = next_tile(tn);
      const TileInfo in2 = tile_info(min(tb, last));
      __builtin_amdgcn_sched_barrier(0);
      compute(rb, ib, full);
      ib = in2;
    }
    if (final_in_b) compute(rb, ib, masked);
    else compute(ra, ia, masked);
  }

  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  const bool wave_bad = __ballot(pid_bad) != 0;
  if (wave_bad) m_run = qnan();  // a bad page poisons the unit: NaN weights below

  // ---- combine the waves: lane (grp, li) holds d = 16*b8 + 4*grp + r4
  if (li < G) {
#pragma unroll
    for (int b8 = 0; b8 < 8; ++b8)
      *reinterpret_cast<f32x4*>(&s_o[w][li][16 * b8 + 4 * grp]) = oacc[b8];
    if (grp == 0) {
      s_m[w][li] = m_run;
      s_l[w][li] = l_run;
    }
  }
  __syncthreads();
  if (tid < G) {
    // a NaN wave max (a bad page) makes the unit's max NaN: fmaxf would skip
    // it, and a range whose waves are all bad would then read as empty (-inf)
    // and be dropped by the combine instead of poisoning the unit
    float M = neg_inf();
    bool nan_m = false;
    for (int ww = 0; ww < kWaves; ++ww) {
      const float mw = s_m[ww][tid];
      nan_m |= mw != mw;
      M = fmaxf(M, mw);
    }
    if (nan_m) M = qnan();
    float L = 0.0f;
    for (int ww = 0; ww < kWaves; ++ww) {
      const float mw = s_m[ww][tid];
      const float wt = mw == neg_inf() ? 0.0f : exp2_fast(mw - M);
      s_m[ww][tid] = wt;  // becomes the wave's weight
      L += wt * s_l[ww][tid];
    }
    s_fm[tid] = M;
    s_fl[tid] = L;
  }
  if (lane == 0 && wave_bad) atomicOr(a.err_flags, KF_EFLAG_BAD_PAGE);  // whichever wave saw it
  __syncthreads();
  if (!work) return;  // after the workgroup's last barrier

  if (nchunks == 1) {
    for (int e = tid; e < G * kDim; e += kThreads) {
      const int h = e / kDim, d = e % kDim;
      float O = 0.0f;
#pragma unroll
      for (int ww = 0; ww < kWaves; ++ww) O += s_m[ww][h] * s_o[ww][h][d];
      a.o_part[((size_t)r * Hq + hq0 + h) * kDim + d] = O / s_fl[h];
    }
    if (tid < G)
      a.lse_part[(size_t)r * Hq + hq0 + tid] = (s_fm[tid] + __log2f(s_fl[tid])) * kLn2;
    return;
  }
  // chunked unit: unnormalised output and (max, sum) of this page range
  const size_t rec = ((size_t)u * H + g) * a.max_chunks + c;
  for (int e = tid; e < G * kDim; e += kThreads) {
    const int h = e / kDim, d = e % kDim;
    float O = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) O += s_m[ww][h] * s_o[ww][h][d];
    a.ws_o[(rec * G + h) * kDim + d] = O;
  }
  if (tid < G) {
    a.ws_ml[(rec * G + tid) * 2] = s_fm[tid];
    a.ws_ml[(rec * G + tid) * 2 + 1] = s_fl[tid];
  }
}

// The dispatch order of a split launch of several rounds.  The hardware
// deals the workgroups of a launch in order over the XCDs and, within an
// XCD, round-robin over its shader engines, and an XCD stops dealing at a
// workgroup whose engine has no free slot: a run of long ranges on one
// engine then idles the others.  Work items (launch position u, KV head,
// range) are therefore listed largest range first (64 size classes), so
// neighbouring workgroups hold ranges of about the same length, and units
// that need no range (empty or bad routes) keep one item for their outputs.
// Which workgroup computes an item does not change any result.  One
// workgroup; the order within a size class follows LDS atomics.  Up to
// kOrderLdsUnits units keep their range count and class in LDS between the
// two passes (more read their routes again).
constexpr int kOrderLdsUnits = 16384;
__global__ __launch_bounds__(1024) void order_kernel(PartialArgs a) {
  __shared__ uint32_t s_count[kOrderBuckets];
  __shared__ uint32_t s_next[kOrderBuckets];
  __shared__ uint16_t s_k[kOrderLdsUnits];
  __shared__ uint8_t s_cls[kOrderLdsUnits];
  const int tid = threadIdx.x, H = a.num_kv_heads, U = a.num_units_routes;
  const bool keep = U <= kOrderLdsUnits;
  if (tid < kOrderBuckets) s_count[tid] = 0;
  __syncthreads();
  // ranges of unit u and the size class of its ranges (0: the largest)
  auto unit = [&](int u, int& k, int& cls) {
    const int r = a.route_list ? a.route_list[u] : u;
    k = 1;
    int size = 0;
    if (r >= 0 && r < a.num_routes) {
      const RouteView rv = read_route(a, r);
      if (!rv.bad && rv.npages > 0) {
        k = (rv.npages + a.chunk_pages - 1) / a.chunk_pages;
        size = (rv.npages + k - 1) / k;
      }
    }
    const int64_t q = (int64_t)size * kOrderBuckets / ((int64_t)a.chunk_pages + 1);
    cls = kOrderBuckets - 1 - (int)(q < kOrderBuckets - 1 ? q : kOrderBuckets - 1);
  };
  for (int u = tid; u < U; u += blockDim.x) {
    int k, cls;
    unit(u, k, cls);
    atomicAdd(&s_count[cls], (uint32_t)(k * H));
    if (keep) {
      s_k[u] = (uint16_t)k;   // k <= max_chunks <= 65535
      s_cls[u] = (uint8_t)cls;
    }
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (int b = 0; b < kOrderBuckets; ++b) {
      s_next[b] = run;
      run += s_count[b];
    }
    a.order[0] = run;
    a.order[1] = 0;
  }
  __syncthreads();
  for (int u = tid; u < U; u += blockDim.x) {
    int k, cls;
    if (keep) {
      k = s_k[u];
      cls = s_cls[u];
    } else {
      unit(u, k, cls);
    }
    const uint32_t pos = atomicAdd(&s_next[cls], (uint32_t)(k * H));
    for (int g = 0; g < H; ++g)
      for (int c = 0; c < k; ++c) {
        const size_t i = pos + (size_t)g * k + c;
        a.order[2 + 2 * i] = (uint32_t)u;
        a.order[3 + 2 * i] = ((uint32_t)g << 16) | (uint32_t)c;
      }
  }
}

// Combine the chunk partials of each chunked (route, KV head) in chunk order.
// Wave w reduces heads w, w+4, ...: its lanes read up to 64 chunks' (max,
// sum) at once; then every thread sums its output elements over the chunks
// in chunk order, four chunks' loads in flight at a time.
__global__ __launch_bounds__(kThreads) void combine_kernel(PartialArgs a) {
  __shared__ float s_fm[KF_MAX_GROUP];
  __shared__ float s_fl[KF_MAX_GROUP];
  const int g = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int G = a.group, Hq = a.num_q_heads, H = a.num_kv_heads;
  const int r = a.route_list ? a.route_list[u] : u;
  if (r < 0 || r >= a.num_routes) return;  // flagged by partial_kernel
  const RouteView rv = read_route(a, r);
  if (rv.bad || rv.npages == 0) return;  // written by partial_kernel
  const int nchunks = (rv.npages + a.chunk_pages - 1) / a.chunk_pages;
  if (nchunks == 1) return;              // written by partial_kernel
  const size_t rec0 = ((size_t)u * H + g) * a.max_chunks;
  for (int h = w; h < G; h += kWaves) {
    float M = neg_inf();
    for (int c = lane; c < nchunks; c += 64) M = fmaxf(M, a.ws_ml[((rec0 + c) * G + h) * 2]);
    for (int m = 32; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m));
    float L = 0.0f;
    for (int c = lane; c < nchunks; c += 64) {
      const float mc = a.ws_ml[((rec0 + c) * G + h) * 2];
      const float lc = a.ws_ml[((rec0 + c) * G + h) * 2 + 1];
      L += mc == neg_inf() ? 0.0f : exp2_fast(mc - M) * lc;
    }
    for (int m = 32; m >= 1; m >>= 1) L += __shfl_xor(L, m);
    if (lane == 0) {
      s_fm[h] = M;
      s_fl[h] = L;
    }
  }
  __syncthreads();
  const int hq0 = g * G;
  for (int e = tid; e < G * kDim; e += kThreads) {
    const int h = e / kDim, d = e % kDim;
    const float M = s_fm[h];
    float O = 0.0f;
#pragma unroll 4
    for (int c = 0; c < nchunks; ++c) {
      const float mc = a.ws_ml[((rec0 + c) * G + h) * 2];
      const float oc = a.ws_o[((rec0 + c) * G + h) * kDim + d];
      O += mc == neg_inf() ? 0.0f : exp2_fast(mc - M) * oc;
    }
    a.o_part[((size_t)r * Hq + hq0 + h) * kDim + d] = O / s_fl[h];
  }
  if (tid < G) a.lse_part[(size_t)r * Hq + hq0 + tid] = (s_fm[tid] + __log2f(s_fl[tid])) * kLn2;
}

// ------------------------------------------------------------------- gather
// Test export: the resident tokens of one route copied out through the same
// route checks (read_route) and page lookup as the attention kernels.  Block
// p copies route-local page p: out[j][g][:] for j = 16 p + slot.
template <class T>
__global__ __launch_bounds__(256) void gather_kernel(PartialArgs a, int route, int max_tokens,
                                                     T* out_k, T* out_v) {
  const int p = blockIdx.x, tid = threadIdx.x, H = a.num_kv_heads;
  const RouteView rv = read_route(a, route);
  if (rv.bad) {
    if (p == 0 && tid == 0) atomicOr(a.err_flags, KF_EFLAG_BAD_ROUTE);
    return;
  }
  const int n = min(rv.n, max_tokens);
  if (p * kPage >= n) return;
  const int pid = a.page_ids[rv.base + p];
  if (pid < 0 || pid >= a.num_pages) {
    if (tid == 0) atomicOr(a.err_flags, KF_EFLAG_BAD_PAGE);
    return;
  }
  const T* kp = static_cast<const T*>(a.k_pool);
  const T* vp = static_cast<const T*>(a.v_pool);
  for (int e = tid; e < H * kPage * kDim; e += blockDim.x) {
    const int g = e / (kPage * kDim), slot = (e / kDim) % kPage, d = e % kDim;
    const int j = p * kPage + slot;
    if (j >= n) continue;
    const size_t head = pool_slice(pid, g, H, a.num_pages, a.head_major);
    out_k[((size_t)j * H + g) * kDim + d] = kp[(head * kPage + slot) * kDim + d];
    out_v[((size_t)j * H + g) * kDim + d] = vp[(head * kDim + d) * kPage + slot];
  }
}

// -------------------------------------------------------------------- merge
// The append decision of sequence b in a fused step, with append_kernel's
// checks and flags: 0 = no append, 1 = appended, else an error flag.
__device__ __forceinline__ int tail_append_status(const MergeArgs& a, int b, int& r) {
  r = a.tail_route[b];
  if (r < 0) return 0;
  if (r >= a.num_routes) return KF_EFLAG_BAD_ROUTE << 8;
  const int32_t* rp = reinterpret_cast<const int32_t*>(a.routes + r);
  const int seq = rp[0], tb = rp[2], te = rp[3], base = rp[4], cap = rp[5];
  const int j = te - tb;
  if (seq != b || j < 0) return KF_EFLAG_BAD_ROUTE << 8;
  if (j / kPage >= cap) return KF_EFLAG_TAIL_FULL << 8;
  if (base < 0 || (int64_t)base + j / kPage >= a.num_page_ids) return KF_EFLAG_BAD_ROUTE << 8;
  const int pid = a.page_ids[base + j / kPage];
  if (pid < 0 || pid >= a.num_pages) return KF_EFLAG_BAD_PAGE << 8;
  return 1;
}

// One wave per (query head, sequence); lane holds dims 2*lane, 2*lane+1.
// In a fused step, wave (0, b) also advances sequence b's tail.
__global__ __launch_bounds__(64) void merge_kernel(MergeArgs a) {
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int Hq = a.num_q_heads;
  if (a.tail_route && h == 0 && lane == 0) {
    int r = 0;
    const int st = tail_append_status(a, b, r);
    if (st == 1)
      a.routes[r].tok_end += 1;  // no other wave of this launch reads it
    else if (st)
      atomicOr(a.err_flags, st >> 8);
  }
  const int r0 = a.seq_route_begin[b], r1 = a.seq_route_begin[b + 1];
  float2* out = reinterpret_cast<float2*>(a.out + ((size_t)b * Hq + h) * kDim) + lane;
  float* lse_out = a.lse_out + (size_t)b * Hq + h;
  if (r0 < 0 || r1 < r0 || r1 > a.num_routes) {
    *out = make_float2(qnan(), qnan());
    if (lane == 0) {
      *lse_out = qnan();
      if (h == 0) atomicOr(a.err_flags, KF_EFLAG_BAD_ROUTE);
    }
    return;
  }
  constexpr float kLog2e = 1.44269504088896340736f;
  // lane i reads the lse of routes r0 + i, r0 + i + 64, ...
  const int n = r1 - r0;
  float M = neg_inf();
  bool nan_seen = false;
  for (int i = lane; i < n; i += 64) {
    const float l = a.lse_part[(size_t)(r0 + i) * Hq + h];
    nan_seen |= l != l;
    M = fmaxf(M, l);
  }
  for (int m = 32; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m));
  const bool any_nan = __ballot(nan_seen) != 0;
  if (any_nan || M == neg_inf()) {
    const float v = any_nan ? qnan() : 0.0f;
    *out = make_float2(v, v);
    if (lane == 0) *lse_out = any_nan ? qnan() : neg_inf();
    return;
  }
  // routes in order; route base + j's weight comes from lane j
  float L = 0.0f, o0 = 0.0f, o1 = 0.0f;
  for (int base = 0; base < n; base += 64) {
    const int i = base + lane;
    const float wl = i < n ? exp2_fast((a.lse_part[(size_t)(r0 + i) * Hq + h] - M) * kLog2e) : 0.0f;
    const int cnt = min(64, n - base);
    const float2* ob = reinterpret_cast<const float2*>(a.o_part + ((size_t)(r0 + base) * Hq + h) * kDim) + lane;
    const size_t rs = (size_t)Hq * kDim / 2;  // float2 elements from one route's row to the next
    int j = 0;
    for (; j + 4 <= cnt; j += 4) {  // four routes' loads in flight, summed in route order
      float wr[4];
      float2 v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        wr[k] = __shfl(wl, j + k);
        v[k] = ob[(j + k) * rs];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        L += wr[k];
        o0 += wr[k] * v[k].x;
        o1 += wr[k] * v[k].y;
      }
    }
    for (; j < cnt; ++j) {
      const float wr = __shfl(wl, j);
      const float2 v = ob[j * rs];
      L += wr;
      o0 += wr * v.x;
      o1 += wr * v.y;
    }
  }
  *out = make_float2(o0 / L, o1 / L);
  if (lane == 0) *lse_out = M + __logf(L);
}

template <bool FP8, int UPW>
hipError_t launch_partial_kernel(const PartialArgs& a, dim3 grid, hipStream_t stream) {
  if (a.head_major)
    hipLaunchKernelGGL(HIP_KERNEL_NAME(partial_kernel<FP8, UPW, true>), grid, dim3(kThreads * UPW), 0,
                       stream, a);
  else
    hipLaunchKernelGGL(HIP_KERNEL_NAME(partial_kernel<FP8, UPW, false>), grid, dim3(kThreads * UPW), 0,
                       stream, a);
  return hipGetLastError();
}

}  // namespace

// ------------------------------------------------------------------ scratch
// Chunk partials of kf_decode_step_no_alloc: a fixed array in device memory
// that the runtime sets up with the code object on each device, so that the
// call allocates nothing.  Host code never uses the array's name as an
// address: the per-device address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[KF_SCRATCH_BYTES];

namespace {
constexpr int kScratchDevices = 64;
std::atomic<void*> g_scratch_ptr[kScratchDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

hipError_t launch_append(const AppendArgs& a, bool fp8, hipStream_t stream) {
  if (a.num_seqs == 0) return hipSuccess;
  if (fp8)
    hipLaunchKernelGGL(append_kernel<true>, dim3(a.num_seqs), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(append_kernel<false>, dim3(a.num_seqs), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_partial(const PartialArgs& a, bool fp8, hipStream_t stream) {
  if (a.num_units_routes == 0) return hipSuccess;
  if (!fp8 && a.units_per_wg == 2)
    return launch_partial_kernel<false, 2>(a, dim3(1, a.num_kv_heads, (a.num_units_routes + 1) / 2),
                                           stream);
  const dim3 grid(a.max_chunks, a.num_kv_heads, a.num_units_routes);
  if (a.order) {
    hipLaunchKernelGGL(order_kernel, dim3(1), dim3(1024), 0, stream, a);
    const hipError_t eo = hipGetLastError();
    if (eo != hipSuccess) return eo;
  }
  hipError_t e = fp8 ? launch_partial_kernel<true, 1>(a, grid, stream)
                     : launch_partial_kernel<false, 1>(a, grid, stream);
  if (e != hipSuccess || a.max_chunks == 1) return e;
  hipLaunchKernelGGL(combine_kernel, dim3(a.num_kv_heads, a.num_units_routes), dim3(kThreads), 0,
                     stream, a);
  return hipGetLastError();
}

hipError_t launch_gather(const PartialArgs& a, bool fp8, int route, int max_tokens, void* out_k,
                         void* out_v, hipStream_t stream) {
  const int blocks = (max_tokens + kPage - 1) / kPage;
  if (blocks == 0) return hipSuccess;
  if (fp8)
    hipLaunchKernelGGL(gather_kernel<uint8_t>, dim3(blocks), dim3(256), 0, stream, a, route,
                       max_tokens, static_cast<uint8_t*>(out_k), static_cast<uint8_t*>(out_v));
  else
    hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(blocks), dim3(256), 0, stream, a, route,
                       max_tokens, static_cast<uint16_t*>(out_k), static_cast<uint16_t*>(out_v));
  return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t stream) {
  if (a.num_seqs == 0 || a.num_q_heads == 0) return hipSuccess;
  hipLaunchKernelGGL(merge_kernel, dim3(a.num_q_heads, a.num_seqs), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace kf
