// Sparse mixed-precision SwiGLU FFN for one token in one launch (Sec. 1 and
// Sec. 5.2: only the active neurons are computed, each at its precision).
//
//   y += sum_i silu(<g_i, x>) * <u_i, x> * d_i
//
// The work is a list of equal-sized tasks, one per workgroup (8 sixteen-byte
// loads per lane of a 256-thread workgroup, all issued at once):
//
//   h tasks     gate/up dot products of a few neurons of one tier ("units" of
//               d bytes, one or more per wave), h_i = silu(a_i) * b_i, each
//               published as one 64-bit word (call tag, h_i).
//   down tasks  a 512-column slice of y over a run of neurons of one tier:
//               a lane owns 32 columns of one neuron per round; lanes 16 and
//               32 apart share columns and are folded by lane swaps, the
//               waves through LDS, and one fp32 atomic add per column adds
//               the run into y.
//
// Launch order (= workgroup id): h INT4, h INT8, h FP16, down INT4, down
// INT8, down FP16. A down workgroup issues its loads first and then polls the
// h words of its run, which come from workgroups of lower id; on each XCD
// workgroups are dispatched in id order and an h workgroup waits for
// nothing, so every producer runs. The hardware dispatcher replaces each
// finished workgroup at once, so the down loads stream behind the gate/up
// loads without a second launch. The poll is bounded anyway: past the limit
// it sets the layer's status word and takes h = 0. Six workgroups share a CU
// at d = 8192 (76 VGPRs), so enough loads are in flight and the
// dequantization of one workgroup overlaps the loads of the others.
//
// Call tag: the grid has a fixed size per layer (the most tasks a plan of
// the layer can need; workgroups past the plan's tasks exit), and workgroup
// b adds 1 to its own 64-bit counter gen[b] on every call, so all of them
// read the same count E and tag the call E + 1 without a host argument (the
// launch can be captured in a graph and replayed) and without two
// workgroups touching one counter. A word is written and read with single
// agent-scope atomic accesses, so no fence is needed and no word of an
// earlier call is ever taken.
//
// Dequantization is exact and cheap: INT8 / INT4 codes are shifted to
// offset binary (q + 128, q + 8) and placed, by byte permutes or masks, into
// fp16 lanes as denormals n * 2^-24, which v_fma_mix_f32 multiplies exactly
// (by an fp16 x element or an fp32 coefficient) and adds with one rounding.
// The offset comes back out as 128 (or 8) times the sum of x over the chunk
// (h tasks, sums staged in LDS once) or times the sum of the neuron
// coefficients (down tasks), and 2^24 is folded into the scale. (The dot2
// instruction is not used on the offset codes: it does not round its sum to
// nearest, and the offset would magnify its error.)
//
// Padding lanes and invalid slots read slot n_slots, which is all zeros, so
// no load sits under a per-lane branch; every task kind issues the same
// number of loads, so the compiler's wait counts do not depend on the kind.
#include "ffn_tasks.h"

namespace m2c {

namespace {

// Record data is read once per call: non-temporal loads keep it from
// evicting what is reused (slot ids, x, h words, scales, the kernel's code).
// Scales stay normal loads: the lanes and slices of a group share them.
typedef uint32_t ntv4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16(const uint8_t* p) {
  const ntv4 v = __builtin_nontemporal_load(reinterpret_cast<const ntv4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint32_t ld2(const uint8_t* p) {
  return *reinterpret_cast<const uint16_t*>(p);
}
__device__ __forceinline__ float lo_f(uint32_t p) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(p & 0xffffu));
}
__device__ __forceinline__ float hi_f(uint32_t p) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(p >> 16));
}

static_assert(kFNPR * kFL <= kWorkSlotPad && kFWaves * kFL <= kWorkSlotPad,
              "slot id reads stay inside the padded work_slot array");

// Unscaled dot products of one 16-byte chunk of INT8 (16 codes) or INT4 (32
// codes) weights with their x elements (x0, x1 / xq: the chunk's x as it sits
// in LDS), offset codes as fp16 denormals: sum of (q + 128) x or (q + 8) x,
// times 2^-24.
__device__ __forceinline__ float chunk_int8(const uint4 v, const uint4 x0, const uint4 x1) {
  const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
  const uint32_t xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
  float t = 0.0f;
#pragma unroll
  for (int u4 = 0; u4 < 4; ++u4) {
    const uint32_t ob = wv[u4] ^ 0x80808080u;  // q + 128
    const uint32_t l = __builtin_amdgcn_perm(0u, ob, 0x0c010c00u);
    const uint32_t h = __builtin_amdgcn_perm(0u, ob, 0x0c030c02u);
    t = fmaf(lo_f(l), lo_f(xv[2 * u4]), t);
    t = fmaf(hi_f(l), hi_f(xv[2 * u4]), t);
    t = fmaf(lo_f(h), lo_f(xv[2 * u4 + 1]), t);
    t = fmaf(hi_f(h), hi_f(xv[2 * u4 + 1]), t);
  }
  return t;
}
// INT4 codes to fp16 lanes by masks alone: nibble n of a word is x element n
// of its 8; nibbles 0 | 4 and, after a shift by 8, 2 | 6 land in the low bits
// of the two fp16 halves (value q + 8), nibbles 1 | 5 and 3 | 7 four bits up
// (16 times that value, still an exact denormal). The two kinds are summed
// apart and joined with an exact 1/16.
struct Nib4 {
  uint32_t p0, p1, p2, p3;  // nibbles (0, 4), (1, 5) x 16, (2, 6), (3, 7) x 16
};
__device__ __forceinline__ Nib4 nibbles(uint32_t w) {
  const uint32_t w8 = w >> 8;
  return {(w ^ 0x88888888u) & 0x000f000fu, (w ^ 0x88888888u) & 0x00f000f0u,
          (w8 ^ 0x88888888u) & 0x000f000fu, (w8 ^ 0x88888888u) & 0x00f000f0u};
}
__device__ __forceinline__ float chunk_int4(const uint4 v, const uint4 (&xq)[4]) {
  const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
  float ta = 0.0f, tb = 0.0f;  // codes at their value, codes at 16 times it
#pragma unroll
  for (int u4 = 0; u4 < 4; ++u4) {
    const uint32_t xw[4] = {xq[u4].x, xq[u4].y, xq[u4].z, xq[u4].w};  // x[8 u4 .. 8 u4 + 7]
    const Nib4 n = nibbles(wv[u4]);
    ta = fmaf(lo_f(n.p0), lo_f(xw[0]), ta);
    ta = fmaf(hi_f(n.p0), lo_f(xw[2]), ta);
    tb = fmaf(lo_f(n.p1), hi_f(xw[0]), tb);
    tb = fmaf(hi_f(n.p1), hi_f(xw[2]), tb);
    ta = fmaf(lo_f(n.p2), lo_f(xw[1]), ta);
    ta = fmaf(hi_f(n.p2), lo_f(xw[3]), ta);
    tb = fmaf(lo_f(n.p3), hi_f(xw[1]), tb);
    tb = fmaf(hi_f(n.p3), hi_f(xw[3]), tb);
  }
  return fmaf(tb, 0.0625f, ta);
}

__device__ __forceinline__ unsigned long long load_word(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The first kFT words are not used: with h at offset 0 the register
// allocator of hipcc (ROCm 7.2) spills a VGPR in the down path of some
// instances, and this layout compiles without scratch for every K.
struct FShared {
  int unused[kFT];
  float h[kFT];                // down task: the h values of its neurons
  float2 ab[kFWaves * kFL];    // h task: per-unit gate / up sums
};

// Sum over the four lane groups of a wave (lanes 16 apart hold the same
// columns of four neurons): 16 column sums per lane in, 4 out. Lanes l and
// l + 32 swap halves of their sums (the lower lane keeps columns 0..7, the
// upper 8..15), then lanes l and l + 16 within each half do the same with what
// is left, so lane l ends with columns 4 (l / 16) .. 4 (l / 16) + 3.
__device__ __forceinline__ void wave_fold16(const float (&acc)[16], float (&out)[4]) {
  float a[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[e]),
                                                    __float_as_uint(acc[8 + e]), false, false);
    a[e] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a[e]),
                                                    __float_as_uint(a[4 + e]), false, false);
    out[e] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
}

// Cross-wave sums of a down task: wave w stores the 32 columns of lane group
// i (lane % 16) as row i of its [16][36] block (the 4-word pad spreads the 64
// lanes' 16-byte stores over every bank); thread c then adds column c of the
// kFWaves blocks.
constexpr int kFRow = 36;
constexpr int kFBlock = (kFSW / 32) * kFRow;
constexpr size_t kFFoldBytes = (size_t)kFWaves * kFBlock * 4;

// Dynamic LDS: x [d/8] | -128 * sums of 16 elements [d/16] | -8 * sums of 32
// [d/32] for h tasks; the same bytes hold the fold of a down task.
inline size_t fused_lds_bytes(int d) {
  const size_t xb = (size_t)d * 2 + (size_t)d / 16 * 4 + (size_t)d / 32 * 4;
  return xb > kFFoldBytes ? xb : kFFoldBytes;
}

// What a task needs besides its slot ids: the slot arena and its zero slot,
// the pool of the task's tier (byte offset of its first slot, first slot id,
// slot count, record stride) and the task's work items.
struct FTaskArgs {
  const uint8_t* slots;
  uint32_t zero;
  uint32_t tb, tf, tc, ts;
  int d;
  int lo, n;  // first work item, items
  int slice;  // down task: column slice
};

// Byte offset of the record in slot v when `ok` and v lies in the task's
// pool, else of the zero slot (every record byte there is 0). Offsets stay
// below 4 GiB (checked at launch), so every address is the arena base plus
// one 32-bit register.
__device__ __forceinline__ uint32_t rec_of(const FTaskArgs& a, int v, bool ok) {
  const uint32_t i = (uint32_t)(v - (int)a.tf);
  return ok && i < a.tc ? a.tb + i * a.ts : a.zero;
}

// An h task of tier TIER (one code path per tier and kind: every branch
// below is on a compile-time value or a wave-uniform one, and no path shares
// blocks with another, so the loads of a task go out back to back).
//   loads: x (from the caches, ahead of the records), then kFL 16-byte record
//   loads per lane and, for INT8 / INT4, the group scale of each.
//   x into LDS with the chunk sums for the code offsets, the gate / up sums
//   of every unit, then h_i = silu(a_i) b_i per neuron as a (call tag, h)
//   word. A unit whose slot id is past the task or outside the pool reads the
//   zero slot, so its sums and h are exactly 0.
template <int K, int TIER, bool EXACT>
__device__ __forceinline__ void h_task(const FTaskArgs& a, const int (&idt)[kFL][4],
                                       const uint16_t* __restrict__ x, uint4* xlds, FShared& sh,
                                       unsigned long long* __restrict__ hw, uint32_t epoch,
                                       int withhold, int tid) {
  constexpr int UW = kFL / K;                             // units per wave
  constexpr int upi = TIER == 3 ? 4 : TIER == 2 ? 2 : 1;  // units per neuron
  constexpr int kXC = 8192 / 16 / kFT;                    // x chunks of 16 values per thread
  static_assert(kXC * kFT * 16 == 8192, "x staging covers d = 8192");
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  // EXACT: d = 1024 K, a unit's rows fill its K loads exactly (every address
  // offset is then a constant)
  const int d = EXACT ? 1024 * K : a.d;
  const uint32_t ud = (uint32_t)d;
  const uint32_t G = ud >> 7;
  const int ncu = d >> 5;  // 16-byte chunks of each row in a unit
  const uint32_t row = TIER == 3 ? 2 * ud : TIER == 2 ? ud : (ud >> 1);
  const uint32_t sbase = TIER == 1 ? 3 * (ud >> 1) : 3 * ud;
  const int nc8 = d >> 3;
  const uint4* x4 = reinterpret_cast<const uint4*>(x);
  uint4 xv[kXC][2];
#ifdef M2C_X_FIRST
#pragma unroll
  for (int k = 0; k < kXC; ++k) {
    const int c = tid + k * kFT;
    xv[k][0] = x4[min(2 * c, nc8 - 1)];
    xv[k][1] = x4[min(2 * c + 1, nc8 - 1)];
  }
#endif
  // unit wu UW + uw of the task sits at table entry (uw / 4) kFNPR + 4 wu + uw % 4
  uint32_t rec[UW];
#pragma unroll
  for (int uw = 0; uw < UW; ++uw)
    rec[uw] = rec_of(a, idt[uw >> 2][uw & 3], (wu * UW + uw) / upi < a.n);
  uint4 v[kFL];
  uint32_t sc[kFL];
  int lane_u = lane;
#pragma unroll
  for (int j = 0; j < kFL; ++j) {
    const int part = (wu * UW + j / K) % upi;
    // per unit, the lane index through an opaque copy: the offsets are
    // recomputed per unit instead of being kept live for the next one
    if (!EXACT && j % K == 0) asm volatile("v_mov_b32 %0, %1" : "=v"(lane_u) : "v"(lane));
    int q = lane_u + 64 * (j % K);
    const bool in = q < 2 * ncu;
    q = in ? q : 2 * ncu - 1;
    const bool up = q >= ncu;
    const uint32_t c = (uint32_t)(part * ncu + (up ? q - ncu : q));
    const uint32_t g = TIER == 2 ? (c >> 3) : (c >> 2);
    v[j] = ld16(a.slots + (in ? rec[j / K] + (up ? row : 0) + 16 * c : a.zero));
    if (TIER != 3)
      sc[j] = ld2(a.slots + (in ? rec[j / K] + sbase + 2 * ((up ? G : 0) + g) : a.zero));
  }
#ifndef M2C_X_FIRST
#pragma unroll
  for (int k = 0; k < kXC; ++k) {
    const int c = tid + k * kFT;
    xv[k][0] = x4[min(2 * c, nc8 - 1)];
    xv[k][1] = x4[min(2 * c + 1, nc8 - 1)];
  }
#endif
  // x into LDS and the chunk sums of this thread's 16 values, while the
  // records are in flight
  uint4* xs = xlds;
  float* nx16 = reinterpret_cast<float*>(xlds + (d >> 3));
  float* nx32 = nx16 + (d >> 4);
#pragma unroll
  for (int k = 0; k < kXC; ++k) {
    const int c = tid + k * kFT;  // chunk of 16 x values
    const bool own = 2 * c < nc8;
    if (own) {
      xs[2 * c] = xv[k][0];
      xs[2 * c + 1] = xv[k][1];
    }
    if (TIER != 3) {
      const uint32_t ws[8] = {xv[k][0].x, xv[k][0].y, xv[k][0].z, xv[k][0].w,
                              xv[k][1].x, xv[k][1].y, xv[k][1].z, xv[k][1].w};
      float sum = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) sum += lo_f(ws[e]) + hi_f(ws[e]);
      const float n16 = -128.0f * sum;
      // -8 * (sum of 32) = (-128 * sum of this 16 - 128 * sum of the neighbour's 16) / 16
      const float other = __int_as_float(
          __builtin_amdgcn_mov_dpp(__float_as_int(n16), 0xB1, 0xF, 0xF, false));
      if (own) nx16[c] = n16;
      if (own && (c & 1) == 0) nx32[c >> 1] = (n16 + other) * 0.0625f;
    }
  }
  __syncthreads();
  // each unit's gate / up sums go to LDS as soon as its loads are done, so
  // only one unit's pair of partial sums is live at a time
  auto unit_done = [&](int uw, float ga, float gb) {
    const float sa = wave_sum(ga), sbv = wave_sum(gb);
    if (lane == 0) sh.ab[w * UW + uw] = make_float2(sa, sbv);
  };
  if (K >= 2 && EXACT) {
    // A unit's rows fill its K loads exactly: load jj < K / 2 of a lane is
    // the gate chunk c and load jj + K / 2 the up chunk c, so the x of c is
    // read from LDS once for both.
#pragma unroll
    for (int uw = 0; uw < UW; ++uw) {
      const int part = (w * UW + uw) % upi;
      float ga = 0.0f, gb = 0.0f;
#pragma unroll
      for (int jj = 0; jj < K / 2; ++jj) {
        const int jg = uw * K + jj, ju = jg + K / 2;
        const int c = part * ncu + lane + 64 * jj;
        float pg, pu;
        if (TIER == 3) {
          const uint4 xc = xs[c];
          pg = dot8_f16(v[jg], xc, 0.0f);
          pu = dot8_f16(v[ju], xc, 0.0f);
        } else if (TIER == 2) {
          const uint4 x0 = xs[2 * c], x1 = xs[2 * c + 1];
          const float o = nx16[c];
          pg = h2f((uint16_t)sc[jg]) * fmaf(chunk_int8(v[jg], x0, x1), kTwo24, o);
          pu = h2f((uint16_t)sc[ju]) * fmaf(chunk_int8(v[ju], x0, x1), kTwo24, o);
        } else {
          uint4 xq[4];
#pragma unroll
          for (int u4 = 0; u4 < 4; ++u4) xq[u4] = xs[4 * c + u4];
          const float o = nx32[c];
          pg = h2f((uint16_t)sc[jg]) * fmaf(chunk_int4(v[jg], xq), kTwo24, o);
          pu = h2f((uint16_t)sc[ju]) * fmaf(chunk_int4(v[ju], xq), kTwo24, o);
        }
        ga += pg;
        gb += pu;
        // one chunk at a time: keeps the x reads of later chunks from being
        // hoisted into registers all at once
        __builtin_amdgcn_sched_barrier(0);
      }
      unit_done(uw, ga, gb);
    }
  } else {
    // the lane index through an opaque copy: the chunk indices below are
    // recomputed instead of being kept live from the address computation
    // across the loads (which costs registers, hence spills)
    int lane_c;
    asm volatile("v_mov_b32 %0, %1" : "=v"(lane_c) : "v"(lane));
    float ga = 0.0f, gb = 0.0f;
#pragma unroll
    for (int j = 0; j < kFL; ++j) {
      const int uw = j / K;
      const int part = (w * UW + uw) % upi;
      int q = lane_c + 64 * (j % K);
      q = q < 2 * ncu ? q : 2 * ncu - 1;
      const bool up = q >= ncu;
      const int c = part * ncu + (up ? q - ncu : q);
      float p;
      if (TIER == 3) {
        p = dot8_f16(v[j], xs[c], 0.0f);
      } else if (TIER == 2) {
        p = h2f((uint16_t)sc[j]) * fmaf(chunk_int8(v[j], xs[2 * c], xs[2 * c + 1]), kTwo24,
                                        nx16[c]);
      } else {
        uint4 xq[4];
#pragma unroll
        for (int u4 = 0; u4 < 4; ++u4) xq[u4] = xs[4 * c + u4];
        p = h2f((uint16_t)sc[j]) * fmaf(chunk_int4(v[j], xq), kTwo24, nx32[c]);
      }
      // lanes past the unit read the zero slot: data 0 (FP16) or scale 0
      ga += up ? 0.0f : p;
      gb += up ? p : 0.0f;
      __builtin_amdgcn_sched_barrier(0);
      if (j % K == K - 1) {
        unit_done(uw, ga, gb);
        ga = gb = 0.0f;
      }
    }
  }
  __syncthreads();
  if (tid < a.n) {
    float sa = sh.ab[tid * upi].x, sbv = sh.ab[tid * upi].y;
#pragma unroll
    for (int u = 1; u < upi; ++u) {
      sa += sh.ab[tid * upi + u].x;
      sbv += sh.ab[tid * upi + u].y;
    }
    const float h = silu_mul(sa, sbv);
    const unsigned long long word =
        ((unsigned long long)epoch << 32) | (unsigned long long)__float_as_uint(h);
    if (withhold == 0)  // test support withholds the word to drive the give-up path
      __hip_atomic_store(hw + a.lo + tid, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Down projection of a down task: columns 16 * HALF .. 16 * HALF + 15 of the
// lane's 32, for every neuron of the task (the two halves share the loaded
// data and keep only 16 accumulators live). csum: sum of the lane's
// coefficients, for the offset of INT8 / INT4 codes. sc[q]: the group scale
// of the lane's neuron in round q.
template <int HALF, int TIER>
__device__ __forceinline__ void compute_dn_half(const uint4 (&v)[kFL], const uint32_t (&sc)[kFL],
                                                const float* s_h, int tid, float (&acc)[16]) {
  const int r = tid / kFLPN;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
  if (TIER == 3) {
    // 4 loads per neuron and round, 8 columns each: this half is loads 2H, 2H+1
#pragma unroll
    for (int q = 0; q < kDnRounds3; ++q) {
      const float c = s_h[q * kFNPR + r];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const uint4 vv = v[4 * q + 2 * HALF + e];
        const uint32_t ws[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc[8 * e + 2 * u] = fmaf(c, lo_f(ws[u]), acc[8 * e + 2 * u]);
          acc[8 * e + 2 * u + 1] = fmaf(c, hi_f(ws[u]), acc[8 * e + 2 * u + 1]);
        }
      }
    }
  } else if (TIER == 2) {
    // 2 loads per neuron and round, 16 columns each: this half is load H
    float csum = 0.0f;
#pragma unroll
    for (int q = 0; q < kDnRounds2; ++q) {
      const float c = s_h[q * kFNPR + r] * h2f((uint16_t)sc[q]);
      csum += c;
      const float cs = c * kTwo24;
      const uint4 vv = v[2 * q + HALF];
      const uint32_t ws[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t ob = ws[u] ^ 0x80808080u;
        const uint32_t l = __builtin_amdgcn_perm(0u, ob, 0x0c010c00u);
        const uint32_t h = __builtin_amdgcn_perm(0u, ob, 0x0c030c02u);
        acc[4 * u] = fmaf(cs, lo_f(l), acc[4 * u]);
        acc[4 * u + 1] = fmaf(cs, hi_f(l), acc[4 * u + 1]);
        acc[4 * u + 2] = fmaf(cs, lo_f(h), acc[4 * u + 2]);
        acc[4 * u + 3] = fmaf(cs, hi_f(h), acc[4 * u + 3]);
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = fmaf(-128.0f, csum, acc[e]);
  } else {
    // 1 load per neuron and round, 32 columns: this half is words 2H, 2H+1
    float csum = 0.0f;
#pragma unroll
    for (int q = 0; q < kDnRounds1; ++q) {
      const float c = s_h[q * kFNPR + r] * h2f((uint16_t)sc[q]);
      csum += c;
      const float cs = c * kTwo24;
      const uint32_t ws[2] = {HALF ? v[q].z : v[q].x, HALF ? v[q].w : v[q].y};
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        // column 8 u + e is nibble e; odd columns sum 16 times their value.
        // Nibbles 0..3 first, then 4..7 (after the barrier): fewer codes live.
        const uint32_t w = ws[u] ^ 0x88888888u;
        const uint32_t p0 = w & 0x000f000fu, p1 = w & 0x00f000f0u;
        acc[8 * u + 0] = fmaf(cs, lo_f(p0), acc[8 * u + 0]);
        acc[8 * u + 4] = fmaf(cs, hi_f(p0), acc[8 * u + 4]);
        acc[8 * u + 1] = fmaf(cs, lo_f(p1), acc[8 * u + 1]);
        acc[8 * u + 5] = fmaf(cs, hi_f(p1), acc[8 * u + 5]);
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t w8 = w >> 8;
        const uint32_t p2 = w8 & 0x000f000fu, p3 = w8 & 0x00f000f0u;
        acc[8 * u + 2] = fmaf(cs, lo_f(p2), acc[8 * u + 2]);
        acc[8 * u + 6] = fmaf(cs, hi_f(p2), acc[8 * u + 6]);
        acc[8 * u + 3] = fmaf(cs, lo_f(p3), acc[8 * u + 3]);
        acc[8 * u + 7] = fmaf(cs, hi_f(p3), acc[8 * u + 7]);
        __builtin_amdgcn_sched_barrier(0);  // one word's codes live at a time
      }
    }
    // exact: the odd columns' sums are 16 times the true ones, rounding included
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = fmaf(acc[e], (e & 1) ? 0.0625f : 1.0f, -8.0f * csum);
  }
}

// A down task of tier TIER: a 512-column slice of y over a run of neurons.
//   loads: kFL 16-byte loads per lane (a wave covers neurons 4 w .. 4 w + 3
//   of every round, lane group lane / 16 its own one, 32 columns per lane)
//   and, for INT8 / INT4, one group scale per round;
//   then the h words of the run (polled, bounded), the column sums per lane,
//   the fold over the wave's lane groups and the waves, one fp32 atomic add
//   per column.
template <int TIER>
__device__ __forceinline__ void dn_task(const FTaskArgs& a, const int (&idt)[kFL][4],
                                        uint4* xlds, FShared& sh,
                                        const unsigned long long* __restrict__ hw,
                                        int32_t* __restrict__ status, float* __restrict__ y,
                                        uint32_t epoch, int withhold, int tid) {
  constexpr int lnv = TIER == 3 ? 2 : TIER == 2 ? 1 : 0;  // log2 loads per neuron and round
  constexpr int R = kFL >> lnv;                            // rounds
  const int lane = tid & 63;
  const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t ud = (uint32_t)a.d;
  const uint32_t G = ud >> 7;
  const uint32_t col = (uint32_t)(a.slice * kFSW + 32 * (tid % kFLPN));
  const bool colok = col < ud;
  const uint32_t dbase = TIER == 3 ? 4 * ud + 2 * col : TIER == 2 ? 2 * ud + col : ud + (col >> 1);
  const uint32_t sbase = (TIER == 1 ? 3 * (ud >> 1) : 3 * ud) + 4 * G + 2 * (col >> 7);
  const int sub = lane >> 4;
  uint32_t rec[R];
#pragma unroll
  for (int q = 0; q < R; ++q) {
    uint32_t rr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) rr[i] = rec_of(a, idt[q][i], q * kFNPR + 4 * wu + i < a.n);
    rec[q] = sub == 0 ? rr[0] : sub == 1 ? rr[1] : sub == 2 ? rr[2] : rr[3];
  }
  uint4 v[kFL];
  uint32_t sc[kFL];
#pragma unroll
  for (int j = 0; j < kFL; ++j) {
    const int q = j >> lnv, e = j & ((1 << lnv) - 1);
    v[j] = ld16(a.slots + (colok ? rec[q] + dbase + 16 * e : a.zero));
    if (TIER != 3 && e == 0) sc[q] = ld2(a.slots + (colok ? rec[q] + sbase : a.zero));
  }
  // the h words of the run, polled after every load has been issued
  float h = 0.0f;
  if (tid < a.n) {
    unsigned long long hv = load_word(hw + a.lo + tid);
    const int limit = withhold > 0 ? withhold : kFSpin;
    int spins = 0;
    while ((uint32_t)(hv >> 32) != epoch) {
      if (++spins > limit) {
        atomicOr(status, M2C_STATUS_FFN_WAIT);
        hv = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      hv = load_word(hw + a.lo + tid);
    }
    h = __uint_as_float((uint32_t)hv);
  }
  sh.h[tid] = h;
  __syncthreads();
  // Per half slice: 16 column sums per lane, folded over the wave's four
  // neurons of each round to 4 (columns 4 g .. 4 g + 3 of the half, g =
  // lane / 16); then the waves through LDS and one fp32 atomic add per
  // column. (Each lane stores its own four sums of a half as soon as they
  // are folded: the LDS bytes are not used otherwise by a down task.)
  float* part = reinterpret_cast<float*>(xlds);
  float* row = part + (tid >> 6) * kFBlock + (tid & 15) * kFRow + 4 * ((tid & 63) >> 4);
  {
    float acc[16], o[4];
    compute_dn_half<0, TIER>(v, sc, sh.h, tid, acc);
    wave_fold16(acc, o);
    *reinterpret_cast<float4*>(row) = make_float4(o[0], o[1], o[2], o[3]);
  }
  {
    float acc[16], o[4];
    compute_dn_half<1, TIER>(v, sc, sh.h, tid, acc);
    wave_fold16(acc, o);
    *reinterpret_cast<float4*>(row + 16) = make_float4(o[0], o[1], o[2], o[3]);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kFSW / kFT; ++k) {
    const int c = tid + k * kFT;  // column of the slice
    const float* src = part + (c >> 5) * kFRow + (c & 31);
    float s = 0.0f;
#pragma unroll
    for (int w = 0; w < kFWaves; ++w) s += src[w * kFBlock];
    const int cy = a.slice * kFSW + c;
    if (cy < a.d) atomicAdd(y + cy, s);
  }
}

// Register budget of at least five workgroups per CU (96 VGPRs). At d = 8192
// the code takes 76, so six are resident, which the LDS (21.8 KB per
// workgroup) also allows. Six is the measured optimum there: seven (INT4
// gate / up chunks computed in pairs, 67 VGPRs, no spills) took 14.6 us
// against 14.36, five 15.5. At d = 4096 the code takes 96 (five).
#ifndef M2C_FFN_WAVES_PER_EU
#define M2C_FFN_WAVES_PER_EU 5
#endif
// EXACT: d = 1024 K (constant offsets in the h tasks), a kernel of its own so
// that the register count of the general-d paths does not set its occupancy.
// General d at K = 4 gets a budget of four workgroups per CU: its INT4 h path
// needs 100 VGPRs, and at 96 the compiler spills scale values as they load,
// each spill waiting for every load in flight.
template <int K, bool EXACT>
__global__ __launch_bounds__(kFT) __attribute__((amdgpu_waves_per_eu(
    K == 4 && !EXACT ? 4 : M2C_FFN_WAVES_PER_EU))) void ffn_fused_kernel(
    const uint16_t* __restrict__ x, const int32_t* __restrict__ tasks,
    const int32_t* __restrict__ task_ids, unsigned long long* __restrict__ gen,
    const uint8_t* __restrict__ slots, int d, unsigned long long* __restrict__ hw,
    int32_t* __restrict__ status, float* __restrict__ y, int withhold) {
  // (argument order: what the first round trip needs comes first, inside the
  // preloaded kernel arguments)
  extern __shared__ uint4 xlds[];  // fused_lds_bytes(d)
  __shared__ FShared sh;
  const int tid = threadIdx.x;
  const int t = blockIdx.x;
  // Everything the data loads need sits at addresses that depend on the
  // workgroup id alone (task count, this task's header and its wave's slot
  // ids, the call counter): one round trip of scalar loads before they go out.
  const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t* wp = task_ids + (int64_t)t * kTaskIds + 4 * wu;
  int idt[kFL][4];
#pragma unroll
  for (int q = 0; q < kFL; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) idt[q][i] = __builtin_amdgcn_readfirstlane(wp[q * kFNPR + i]);
  const int n_tasks = tasks[0];
  const uint32_t zero = (uint32_t)tasks[1];
  const int4 hd = reinterpret_cast<const int4*>(tasks + 4)[2 * t];
  const int4 hp = reinterpret_cast<const int4*>(tasks + 4)[2 * t + 1];
  const unsigned long long e0 = gen[t];  // the call count: only this workgroup touches gen[t]
  // (every load above goes out before the first is used; the call count is
  // needed only at the end, and this keeps its load in the first round trip
  // instead of one of its own after the task header)
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::"s"((uint32_t)e0), "s"((uint32_t)(e0 >> 32)));
  const int kind = t < n_tasks ? (hd.x & 0xff) : 0;
  const int tier = (hd.x >> 8) & 0xff;
  if (kind != 1 && kind != 2) {
    if (tid == 0) gen[t] = e0 + 1;  // keep this workgroup's count in step
    return;
  }
  FTaskArgs a;
  a.slots = slots;
  a.zero = zero;
  a.tb = (uint32_t)hp.x;
  a.tf = (uint32_t)hp.y;
  a.tc = (uint32_t)hp.z;
  a.ts = (uint32_t)hp.w;
  a.d = d;
  a.lo = hd.y;
  a.n = hd.z;
  a.slice = hd.w;
  const uint32_t epoch = (uint32_t)e0 + 1u;
  if (kind == 1) {
    if constexpr (EXACT) {
      if (tier == 1)
        h_task<K, 1, true>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
      else if (tier == 2)
        h_task<K, 2, true>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
      else
        h_task<K, 3, true>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
    } else {
      if (tier == 1)
        h_task<K, 1, false>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
      else if (tier == 2)
        h_task<K, 2, false>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
      else
        h_task<K, 3, false>(a, idt, x, xlds, sh, hw, epoch, withhold, tid);
    }
  } else {
    if (tier == 1)
      dn_task<1>(a, idt, xlds, sh, hw, status, y, epoch, withhold, tid);
    else if (tier == 2)
      dn_task<2>(a, idt, xlds, sh, hw, status, y, epoch, withhold, tid);
    else
      dn_task<3>(a, idt, xlds, sh, hw, status, y, epoch, withhold, tid);
  }
  if (tid == 0) gen[t] = e0 + 1;
}

template <int K>
hipError_t launch_fused(m2c_layer* L, const uint16_t* x, const int32_t* tasks, float* y,
                        hipStream_t stream) {
  const int d = L->desc.d_model;
  const size_t lds = fused_lds_bytes(d);
  const int32_t* task_ids = tasks + task_ids_offset(L->ffn_grid) / 4;
  if (K >= 2 && d == 1024 * K)
    hipLaunchKernelGGL((ffn_fused_kernel<K, K >= 2>), dim3(L->ffn_grid), dim3(kFT), lds, stream,
                       x, tasks, task_ids, L->st.ffn_gen, L->slots, d, L->st.ffn_hw, L->st.status,
                       y, L->ffn_withhold);
  else
    hipLaunchKernelGGL((ffn_fused_kernel<K, false>), dim3(L->ffn_grid), dim3(kFT), lds, stream, x,
                       tasks, task_ids, L->st.ffn_gen, L->slots, d, L->st.ffn_hw, L->st.status, y,
                       L->ffn_withhold);
  return hipGetLastError();
}

// The task table of a plan (the single cache unit's plan; the per-tier
// arena's is written with the merge, from the pools' plans).
template <int K>
__global__ __launch_bounds__(256) void ffn_tasks_kernel(const int32_t* __restrict__ counts,
                                                        const int32_t* __restrict__ work_slot,
                                                        int cap, int d, int grid, SlotMap map,
                                                        int32_t* __restrict__ tasks,
                                                        int32_t* __restrict__ task_ids) {
  const FMap m = make_map<K>(counts, cap, d);
  write_task_table<K>(m, grid, map, tasks, task_ids,
                      (int)(blockIdx.x * blockDim.x + threadIdx.x) >> 6,
                      (int)(gridDim.x * blockDim.x) >> 6, [&](int e) { return work_slot[e]; });
}

template <int K>
hipError_t launch_tasks(m2c_layer* L, uint8_t* plan, hipStream_t stream) {
  const m2c_plan_layout& lay = L->layout;
  int32_t* tasks = reinterpret_cast<int32_t*>(plan + lay.ffn_tasks);
  int blocks = (L->ffn_grid + 3) / 4;
  blocks = blocks < 1 ? 1 : blocks > 256 ? 256 : blocks;
  hipLaunchKernelGGL(ffn_tasks_kernel<K>, dim3(blocks), dim3(256), 0, stream,
                     reinterpret_cast<const int32_t*>(plan + lay.counts),
                     reinterpret_cast<const int32_t*>(plan + lay.work_slot), L->cap,
                     L->desc.d_model, L->ffn_grid, L->map, tasks,
                     tasks + task_ids_offset(L->ffn_grid) / 4);
  return hipGetLastError();
}

}  // namespace

int ffn_loads_per_unit(int d) {
  const int kneed = (d + 1023) / 1024;
  return kneed <= 1 ? 1 : kneed <= 2 ? 2 : kneed <= 4 ? 4 : 8;
}

bool ffn_fused_supported(const m2c_layer* L) {
  return L->desc.d_model <= 8192 && L->arena_bytes < ((int64_t)1 << 32);
}

int ffn_fused_grid(int d, int cap, int num_cus) {
  (void)num_cus;
  if (cap <= 0) return 0;
  // h tasks: at most cap / (FP16 neurons per task) + 1 per tier; down tasks:
  // per slice at most cap / (FP16 neurons per run) + 1 per tier
  const int U = kFWaves * (kFL / ffn_loads_per_unit(d));
  const int64_t most = (int64_t)cap / (U / 4) + 3 +
                       (int64_t)((d + kFSW - 1) / kFSW) * (cap / (kDnRounds3 * kFNPR) + 3);
  return (int)most;
}

hipError_t launch_ffn_fused(m2c_layer* L, const uint16_t* x, const uint8_t* plan, float* y,
                            hipStream_t stream) {
  if (L->cap <= 0 || L->ffn_grid <= 0) return hipSuccess;
  const int32_t* tasks = reinterpret_cast<const int32_t*>(plan + L->layout.ffn_tasks);
  switch (ffn_loads_per_unit(L->desc.d_model)) {
    case 1: return launch_fused<1>(L, x, tasks, y, stream);
    case 2: return launch_fused<2>(L, x, tasks, y, stream);
    case 4: return launch_fused<4>(L, x, tasks, y, stream);
    default: return launch_fused<8>(L, x, tasks, y, stream);
  }
}

bool ffn_tasks_used(const m2c_layer* L) {
  return !(L->desc.flags & M2C_FLAG_DETERMINISTIC_FFN) && ffn_fused_supported(L) && L->cap > 0;
}

int64_t ffn_task_table_bytes(int grid) {
  return task_ids_offset(grid) + (int64_t)grid * kTaskIds * 4;
}

hipError_t launch_ffn_tasks(m2c_layer* L, uint8_t* plan, hipStream_t stream) {
  if (!ffn_tasks_used(L) || L->ffn_grid <= 0) return hipSuccess;
  switch (ffn_loads_per_unit(L->desc.d_model)) {
    case 1: return launch_tasks<1>(L, plan, stream);
    case 2: return launch_tasks<2>(L, plan, stream);
    case 4: return launch_tasks<4>(L, plan, stream);
    default: return launch_tasks<8>(L, plan, stream);
  }
}

}  // namespace m2c
