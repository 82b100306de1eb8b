// Attention of a band's queries over the keys/values of the whole image,
// fresh for the band's tokens and stale (from the buffer) for all others
// (patch parallelism with stale activations, §II-B; Algorithm 1).
//
// bf16 path: a flash-style kernel on v_mfma_f32_32x32x16_bf16.  Each
// workgroup owns 128 queries of one (branch, head); each wave 32 of them.
// Scores are formed transposed, S^T = K Q^T, so that a lane owns one query
// column: the running max of the online softmax stays in-lane, and the
// probabilities it holds are directly the B operand of O^T = V^T P^T.
// K tiles ([64 keys][d], rows unpadded) and V^T tiles ([d][64 keys], 16-byte
// chunks XOR-swizzled by row) go global -> LDS with the direct-to-LDS load
// into a ring of three stages, one barrier per tile.  K rows are permuted in
// LDS (bits 2 and 3 of the row swapped) so that the 8 keys of each lane's P
// fragment are contiguous in natural key order.  When the head dimension is
// padded (d = 72 -> 96 rows of O^T), one padding row of V^T holds ones, so
// the PV product also accumulates the softmax denominator.  exp2 runs on
// v_exp_f32 with log2(e)/sqrt(d) folded into the exponent; the running max is
// raised lazily (only past a 2^8 margin), so O is rarely rescaled.  The loop
// runs over 32-key halves of a tile: the MFMAs of the next half's scores are
// issued between the current half's exponentials, then its PV MFMAs.  Built
// without IEEE NaN quieting, so the row max is plain v_max3_f32.
//
// fp32 path (and unsupported shapes): one thread per query, online softmax.
#include "common.h"
#include "kernels.h"

namespace orch {

namespace mfma_attn {
constexpr int BQ = 128, BKV = 64, NSTAGE = 4;

template <int D>
struct Geo {
  static constexpr int NC = (D + 15) / 16;          // 16-dim chunks of S^T = K Q^T
  static constexpr int NS = 2 * NC;                 // MFMAs of one S^T tile
  static constexpr int DV = (D + 31) / 32 * 32;     // rows of O^T, padded to 32
  static constexpr int NT = DV / 32;
  static constexpr bool ONES = DV > D;              // padding row D of V^T holds 1.0
  static constexpr int KROW = 2 * D;                // bytes per K row in LDS
  static constexpr int KCH = KROW / 16;             // 16-byte chunks per K row
  static constexpr bool KSWZ = KCH == 8;            // 128-byte rows: XOR swizzle
  static constexpr int K_BYTES = BKV * KROW;
  static constexpr int K_SPAN = (K_BYTES + 16 + 255) / 256 * 256;  // 16 zero bytes after K
  static constexpr int VROW = 2 * BKV;              // bytes per V^T row
  static constexpr int V_BYTES = D * VROW;
  static constexpr int STAGE = K_SPAN + V_BYTES;
  static constexpr int CONST_OFF = NSTAGE * STAGE;  // V^T rows [D, DV), shared by the stages
  static constexpr int DUMMY_OFF = CONST_OFF + (DV - D) * VROW;  // sink of padding loads
  static constexpr int LDS = DUMMY_OFF + 1024;
  static constexpr int K_LOADS = K_BYTES / 1024;    // 1 KB wave-level loads
  static constexpr int V_LOADS = V_BYTES / 1024;
  // waves 0-1 load K, waves 2-3 V^T, LPW loads each per tile; slots past the
  // tile's loads re-read a valid chunk into the sink, so every wave counts
  // the same number of loads
  static constexpr int LPW = (cmax(K_LOADS, V_LOADS) + 1) / 2;
  static_assert(K_BYTES % 1024 == 0 && V_BYTES % 1024 == 0, "whole 1 KB loads");
  // 16 consecutive K rows at one 16-byte column must hit distinct 4-bank
  // groups: an odd number of chunks per row, or 8 chunks with the swizzle
  static_assert(KCH == 8 || KCH % 2 == 1, "K row layout");
  static_assert(2 * LDS <= 160 * 1024, "two workgroups per CU");
  static_assert(2 * LPW < 16, "loads in flight");
};

// LDS row rho of a K tile holds key kperm(rho): bits 2 and 3 swapped.  The
// S^T accumulator row 8g + 4h + r then belongs to key 16c + 8h + e for the
// P fragment (chunk c, element e) a lane with half h feeds to the PV MFMA,
// i.e. the 8 keys of a lane's fragment are contiguous and V^T stays in
// natural key order.
__device__ __forceinline__ int kperm(int rho) {
  return (rho & ~12) | ((rho & 4) << 1) | ((rho & 8) >> 1);
}

// word 3 of a raw buffer resource (gfx9: 32-bit data format, no swizzle)
constexpr int kBufWord3 = 0x00020000;

// Resource of a wave-uniform buffer; the base and size go through
// readfirstlane so the compiler keeps the descriptor in SGPRs.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, size_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* ub = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, __builtin_amdgcn_readfirstlane((int)bytes),
                                           kBufWord3);
}
}  // namespace mfma_attn

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bf16_mfma_kernel(AttnParams p) {
  // the body uses device-only types (buffer resources); the host pass only
  // needs the launch stub
#if defined(__HIP_DEVICE_COMPILE__)
  using namespace mfma_attn;
  using G = Geo<D>;
  constexpr int NC = G::NC, NS = G::NS, NT = G::NT, LPW = G::LPW;

  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5;
  const int lc = lane & 31;
  // Workgroups go round-robin over the 8 XCDs; the ones of XCD x take the
  // x-th contiguous eighth of the (branch, head, split, query tile) order, so
  // the query tiles that read the same K/V share one L2.
  const int n_qt = (p.n_q + BQ - 1) / BQ;
  const int T = gridDim.x;
  int lb = blockIdx.x;
  if (lb < T / 8 * 8) lb = (lb & 7) * (T / 8) + (lb >> 3);
  const int qt = lb % n_qt;
  const int split = (lb / n_qt) % p.splits;       // key split of this workgroup
  const int pair = lb / (n_qt * p.splits);
  const int head = pair % p.heads, b = pair / p.heads;
  const int q0 = qt * BQ;
  const int H = p.heads * D;
  const int kv_len = p.n_kv / p.splits;           // multiple of BKV (launcher)
  const int kv0 = split * kv_len;
  const int fb = p.fresh_begin, nf = p.n_fresh;

  const bf16* qbase = reinterpret_cast<const bf16*>(p.q) + ((size_t)b * p.heads + head) * p.n_q * D;
  const bf16* ks = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)head * p.n_kv * D;
  const bf16* vs = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)p.n_kv * H + (size_t)head * D * p.n_kv;
  const bf16* kf = ks;
  const bf16* vf = vs;
  const int fn = nf > 0 ? p.fresh_n : p.n_kv;     // token extent of the fresh buffer
  if (nf > 0) {
    kf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs +
         ((size_t)head * fn + p.fresh_off) * D;
    vf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)fn * H +
         (size_t)head * D * fn + p.fresh_off;
  }
  // buffer resources of this (branch, head): out-of-range reads return zero
  const __amdgpu_buffer_rsrc_t rks = buffer_rsrc(ks, (size_t)p.n_kv * D * 2);
  const __amdgpu_buffer_rsrc_t rvs = buffer_rsrc(vs, (size_t)p.n_kv * D * 2);
  const __amdgpu_buffer_rsrc_t rkf = buffer_rsrc(kf, (size_t)(nf > 0 ? nf : p.n_kv) * D * 2);
  const __amdgpu_buffer_rsrc_t rvf =
      buffer_rsrc(vf, ((size_t)(D - 1) * fn + (nf > 0 ? nf : p.n_kv)) * 2);

  // this lane's query (B operand of S^T = K Q^T): Q[q][c*16 + 8h .. +8]
  const int qrow = min(q0 + wave * 32 + lc, p.n_q - 1);
  bf16x8 qf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int d0 = c * 16 + h * 8;
    if (d0 < D) {
      qf[c] = *reinterpret_cast<const bf16x8*>(qbase + (size_t)qrow * D + d0);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[c][e] = (bf16)0.0f;
    }
  }

  // constant LDS (never written by the tile loads): 16 zero bytes after the
  // K rows of every stage, read against zero Q padding by the last chunk of
  // row 63; V^T rows [D, DV): row D ones, the rest zero
  for (int st = tid; st < NSTAGE * 4; st += 256)
    reinterpret_cast<uint32_t*>(smem + (st >> 2) * G::STAGE + G::K_BYTES)[st & 3] = 0u;
  {
    bf16* cpad = reinterpret_cast<bf16*>(smem + G::CONST_OFF);
    for (int i = tid; i < (G::DV - D) * BKV; i += 256) cpad[i] = (bf16)(i < BKV ? 1.0f : 0.0f);
  }

  // This wave's share of a tile's loads.  Waves 0-1 load K: load j = wave +
  // 2 i fills stage bytes [1024 j, +1024), lane slot s = 64 j + lane is row
  // s / KCH, physical chunk s % KCH.  Waves 2-3 load V^T: load j = wave - 2 +
  // 2 i fills K_SPAN + 1024 j, row s / 8, physical chunk s % 8, logical 8-key
  // chunk = physical ^ ((row >> 1) & 7).  off: byte offset of the lane's
  // source from the tile's first key in the stale buffer (the same for fresh
  // K; fresh V^T rows have stride n_fresh).
  const bool kwave = wave < 2;
  const int wl = wave & 1;
  const int nload = kwave ? G::K_LOADS : G::V_LOADS;
  unsigned off[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int j = min(wl + 2 * i, nload - 1);
    const int sl = j * 64 + lane;
    if (kwave) {
      const int rho = sl / G::KCH, pc = sl % G::KCH;
      const int lch = G::KSWZ ? pc ^ ((rho >> 1) & 7) : pc;
      off[i] = (unsigned)(kperm(rho) * D + lch * 8) * 2u;
    } else {
      const int d = sl >> 3, lch = (sl & 7) ^ ((d >> 1) & 7);
      off[i] = (unsigned)(d * p.n_kv + lch * 8) * 2u;
    }
  }
  // V^T row of load slot i (V waves)
  auto vrow = [&](int i) { return (min(wl + 2 * i, nload - 1) * 64 + lane) >> 3; };
  auto dst_of = [&](int st, int i) -> ORCH_LDS void* {
    const int j = wl + 2 * i;
    if (j >= nload) return (ORCH_LDS void*)(smem + G::DUMMY_OFF);
    return (ORCH_LDS void*)(smem + st * G::STAGE + (kwave ? 0 : G::K_SPAN) + j * 1024);
  };
  auto issue = [&](int n0, int st) {
    const bool all_stale = n0 + BKV <= fb || n0 >= fb + nf;
    const bool all_fresh = n0 >= fb && n0 + BKV <= fb + nf;
    if (all_stale) {
      const __amdgpu_buffer_rsrc_t r = kwave ? rks : rvs;
      const unsigned so = __builtin_amdgcn_readfirstlane((unsigned)n0 * (kwave ? 2 * D : 2));
#pragma unroll
      for (int i = 0; i < LPW; ++i) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst_of(st, i), 16, off[i], so, 0, 0);
    } else if (all_fresh) {
      const __amdgpu_buffer_rsrc_t r = kwave ? rkf : rvf;
      const unsigned so = __builtin_amdgcn_readfirstlane((unsigned)(n0 - fb) * (kwave ? 2 * D : 2));
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        const unsigned o = kwave ? off[i] : off[i] - (unsigned)(vrow(i) * (p.n_kv - fn)) * 2u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst_of(st, i), 16, o, so, 0, 0);
      }
    } else {
      // a tile across the band edge: per-lane source (8-key groups are all
      // fresh or all stale: fb, nf % 8 == 0); 32-bit offsets from the
      // uniform bases keep the loop-invariant part small
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        const char* base;
        unsigned bo;
        if (kwave) {
          const int e = off[i] / 2, key = e / D, col = e - key * D;
          const int n = n0 + key;
          const bool fr = (unsigned)(n - fb) < (unsigned)nf;
          base = reinterpret_cast<const char*>(fr ? kf : ks);
          bo = (unsigned)((fr ? n - fb : n) * D + col) * 2u;
        } else {
          const int d = vrow(i), key = off[i] / 2 - d * p.n_kv;
          const int n = n0 + key;
          const bool fr = (unsigned)(n - fb) < (unsigned)nf;
          base = reinterpret_cast<const char*>(fr ? vf : vs);
          bo = (unsigned)(fr ? d * fn + (n - fb) : d * p.n_kv + n) * 2u;
        }
        __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)(base + bo), dst_of(st, i), 16, 0, 0);
      }
    }
  };
  // wait until at most `tiles` tiles of this wave's loads are in flight
  auto wait_tiles = [&](int tiles) {
    if (tiles <= 0) wait_vmcnt<0>();
    else if (tiles == 1) wait_vmcnt<LPW>();
    else wait_vmcnt<2 * LPW>();
  };

  // fragment read offsets: K row sub*32 + lc, logical chunk 2c + h; V^T row
  // t*32 + lc, logical chunk 2c + h (the swizzle depends on lc only).  V^T
  // rows >= D are the shared constant rows.
  int k_rd[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c)
    k_rd[c] = lc * G::KROW + (G::KSWZ ? ((2 * c + h) ^ ((lc >> 1) & 7)) : (2 * c + h)) * 16;
  int v_rd[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) v_rd[c] = lc * G::VROW + ((2 * c + h) ^ ((lc >> 1) & 7)) * 16;
  const bool last_in_pad = (NT - 1) * 32 + lc >= D;   // row of the last O^T tile is padding

  const float scale = 1.4426950408889634f / sqrtf((float)D);  // log2(e) / sqrt(d)
  float m_run = -1e30f, l_run = 0.0f;
  f32x16 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;

  // K fragments of half `sub` (keys [32 sub, +32)) of the tile in stage st
  auto k_frags = [&](int st, int sub, bf16x8(&kf_)[NC]) {
    const char* sk = smem + st * G::STAGE + sub * 32 * G::KROW;
#pragma unroll
    for (int c = 0; c < NC; ++c) kf_[c] = *reinterpret_cast<const bf16x8*>(sk + k_rd[c]);
  };
  // V^T fragment of O^T tile tt and 16-key chunk c of the tile in stage st
  auto v_frag = [&](int st, int tt, int c) {
    const char* src = (tt == NT - 1 && last_in_pad)
                          ? smem + G::CONST_OFF + (tt * 32 + lc - D) * G::VROW + (v_rd[c] - lc * G::VROW)
                          : smem + st * G::STAGE + G::K_SPAN + tt * 32 * G::VROW + v_rd[c];
    return *reinterpret_cast<const bf16x8*>(src);
  };

  // One 32-key half of a tile: scores sc = S^T of keys [32 sub, +32) of the
  // tile in stage st.  With NEXT, the MFMAs of the next half's scores (K
  // fragments kn, result sn) are issued between the exponentials; then
  // O^T += V^T P^T over the half's two 16-key chunks.
  auto half = [&](auto next_c, int st, int sub, const f32x16& sc, int nst, int nsub, f32x16& sn) {
    constexpr bool NEXT = decltype(next_c)::value;
    // online softmax over this lane's query column.  The running max is only
    // raised when some lane's max exceeds it by more than 8 (log2 units):
    // until then exp2(s - m_run) <= 2^8, exact in fp32 and in range for
    // bf16, and O and the denominator keep a common scale, so O is rarely
    // rescaled.
    float mx = fmaxf(sc[0], sc[1]);
#pragma unroll
    for (int r = 2; r < 16; r += 2) mx = fmaxf(mx, fmaxf(sc[r], sc[r + 1]));
    mx = max_xhalf(mx) * scale;   // VALU swap: no LDS round trip behind the fragment reads
    float alpha = 1.0f;
    if (__any(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[tt][r] *= alpha;
    }
    // the next half's K fragments and this half's V^T fragments, issued after
    // the rescale branch (a branch join makes the compiler wait for every LDS
    // read in flight) and consumed behind the exponentials
    bf16x8 kn[NC];
    if constexpr (NEXT) k_frags(nst, nsub, kn);
    bf16x8 vfr[2][NT];
#pragma unroll
    for (int ci = 0; ci < 2; ++ci)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) vfr[ci][tt] = v_frag(st, tt, 2 * sub + ci);
    __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of their uses
    if constexpr (NEXT) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sn[r] = 0.0f;
    }
    float psum = 0.0f;
    bf16x8 pf[2];
    static_for<0, 2>([&](auto cc) {
      constexpr int ci = decltype(cc)::value;
      if constexpr (NEXT) {
#pragma unroll
        for (int c = ci * NC / 2; c < (ci + 1) * NC / 2; ++c)
          sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kn[c], qf[c], sn, 0, 0, 0);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = 4 * (2 * ci + (e >> 2)) + (e & 3);
        const float pv = __builtin_amdgcn_exp2f(fmaf(sc[r], scale, -m_run));
        if constexpr (!G::ONES) psum += pv;
        pf[ci][e] = (bf16)pv;
      }
    });
    if constexpr (!G::ONES) l_run = l_run * alpha + psum;
    // chunk-major, so consecutive MFMAs accumulate into different O^T tiles
#pragma unroll
    for (int ci = 0; ci < 2; ++ci)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
        o[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[ci][tt], pf[ci], o[tt], 0, 0, 0);
  };

  const int NIT = kv_len / BKV;
#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < NIT) issue(kv0 + s * BKV, s);
  wait_tiles(min(NIT - 1, NSTAGE - 2));
  lds_barrier();

  // scores ping-pong between s0 (first halves) and s1 (second halves)
  f32x16 s0, s1;
  bf16x8 kn[NC];
  k_frags(0, 0, kn);   // the first half's scores
#pragma unroll
  for (int r = 0; r < 16; ++r) s0[r] = 0.0f;
#pragma unroll
  for (int c = 0; c < NC; ++c) s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kn[c], qf[c], s0, 0, 0, 0);

  int t = 0;
  for (; t + 1 < NIT; ++t) {
    const int st = t % NSTAGE;
    half(std::true_type{}, st, 0, s0, st, 1, s1);
    // tile t+1 resident; stage (t-1) % NSTAGE is free for tile t+3
    wait_tiles(t + 2 < NIT ? 1 : 0);
    lds_barrier();
    if (t + NSTAGE - 1 < NIT) issue(kv0 + (t + NSTAGE - 1) * BKV, (t + NSTAGE - 1) % NSTAGE);
    half(std::true_type{}, st, 1, s1, (t + 1) % NSTAGE, 0, s0);
  }
  {
    const int st = t % NSTAGE;
    half(std::true_type{}, st, 0, s0, st, 1, s1);
    half(std::false_type{}, st, 1, s1, 0, 0, s0);
  }

  // softmax denominator: the ones row D of O^T (register 4*((D%32)/8) + D%4
  // of tile D/32 on the h == 0 lanes), or the running sum
  float l;
  if constexpr (G::ONES) {
    constexpr int TR = D / 32, RR = 4 * ((D % 32) / 8) + (D % 4);
    static_assert(((D % 32) / 4) % 2 == 0, "ones row on the h == 0 half");
    l = __shfl(o[TR][RR], lc, kWave);
  } else {
    l = l_run + __shfl_xor(l_run, 32, kWave);
  }
  const int q = q0 + wave * 32 + lc;
  if (p.splits > 1) {
    // partial result of this key split: unnormalised O, running max and sum
    if (q < p.n_q) {
      float* orow = p.part_o + (((size_t)split * p.B + b) * p.n_q + q) * H + head * D;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int d = t * 32 + 8 * g + 4 * h;
          if (d < D)
            *reinterpret_cast<float4*>(orow + d) =
                make_float4(o[t][4 * g], o[t][4 * g + 1], o[t][4 * g + 2], o[t][4 * g + 3]);
        }
      if (h == 0)
        p.part_ml[(((size_t)split * p.B + b) * p.heads + head) * p.n_q + q] = make_float2(m_run, l);
    }
    return;
  }
  const float inv = 1.0f / l;
  if (q < p.n_q) {
    bf16* orow = reinterpret_cast<bf16*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = t * 32 + 8 * g + 4 * h;
        if (d < D) {
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(o[t][4 * g + j] * inv);
          *reinterpret_cast<bf16x4*>(orow + d) = v;
        }
      }
  }
#endif
}

// Combine of the key splits: O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s
// (m = max_s m_s, all in the log2 domain of the kernel above).
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p) {
  const int H = p.heads * p.d;
  const size_t row = blockIdx.y;                 // b * n_q + q
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= H) return;
  const int b = (int)(row / p.n_q), q = (int)(row - (size_t)b * p.n_q);
  const int head = col / p.d;
  float m = -1e30f;
  for (int s = 0; s < p.splits; ++s)
    m = fmaxf(m, p.part_ml[(((size_t)s * p.B + b) * p.heads + head) * p.n_q + q].x);
  float num = 0.0f, den = 0.0f;
  for (int s = 0; s < p.splits; ++s) {
    const float2 ml = p.part_ml[(((size_t)s * p.B + b) * p.heads + head) * p.n_q + q];
    const float w = __builtin_amdgcn_exp2f(ml.x - m);
    num += w * p.part_o[((size_t)s * p.B * p.n_q + row) * H + col];
    den += w * ml.y;
  }
  reinterpret_cast<bf16*>(p.out)[row * H + col] = (bf16)(num / den);
}

// ---------------------------------------------------------------------------
// SIMT attention: one thread per (branch, head, query).
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_simt_kernel(AttnParams p) {
  const int q = blockIdx.x * 64 + threadIdx.x;
  const int head = blockIdx.y;
  const int b = blockIdx.z;
  if (q >= p.n_q) return;
  const int H = p.heads * D;
  const T* qv = reinterpret_cast<const T*>(p.q) + (((size_t)b * p.heads + head) * p.n_q + q) * D;
  const T* ks = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)head * p.n_kv * D;
  const T* vs = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)p.n_kv * H +
                (size_t)head * D * p.n_kv;
  const T* kf = nullptr;
  const T* vf = nullptr;
  if (p.n_fresh > 0) {
    kf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs +
         ((size_t)head * p.fresh_n + p.fresh_off) * D;
    vf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.fresh_n * H +
         (size_t)head * D * p.fresh_n + p.fresh_off;
  }
  float qr[D], acc[D];
  const float scale = 1.0f / sqrtf((float)D);
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qr[d] = to_f<T>(qv[d]) * scale;
    acc[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int n = 0; n < p.n_kv; ++n) {
    const int f = n - p.fresh_begin;
    const bool fresh = (unsigned)f < (unsigned)p.n_fresh;
    const T* kr = fresh ? kf + (size_t)f * D : ks + (size_t)n * D;
    float s = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) s = fmaf(qr[d], to_f<T>(kr[d]), s);
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn);
    const float e = expf(s - mn);
    l = l * a + e;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const float v = fresh ? to_f<T>(vf[(size_t)d * p.fresh_n + f]) : to_f<T>(vs[(size_t)d * p.n_kv + n]);
      acc[d] = fmaf(acc[d], a, e * v);
    }
    m = mn;
  }
  T* o = reinterpret_cast<T*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D;
  const float inv = 1.0f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) o[d] = from_f<T>(acc[d] * inv);
}

// ---------------------------------------------------------------------------
bool attention_uses_mfma(int d, int n_kv, int dtype) {
  return dtype == kBF16 && (d == 64 || d == 72) && n_kv % mfma_attn::BKV == 0;
}

template <typename T>
static hipError_t launch_simt(const AttnParams& p, hipStream_t s) {
  dim3 grid(ceil_div(p.n_q, 64), p.heads, p.B);
  switch (p.d) {
    case 32: hipLaunchKernelGGL((attn_simt_kernel<T, 32>), grid, dim3(64), 0, s, p); break;
    case 64: hipLaunchKernelGGL((attn_simt_kernel<T, 64>), grid, dim3(64), 0, s, p); break;
    case 72: hipLaunchKernelGGL((attn_simt_kernel<T, 72>), grid, dim3(64), 0, s, p); break;
    case 80: hipLaunchKernelGGL((attn_simt_kernel<T, 80>), grid, dim3(64), 0, s, p); break;
    case 96: hipLaunchKernelGGL((attn_simt_kernel<T, 96>), grid, dim3(64), 0, s, p); break;
    case 128: hipLaunchKernelGGL((attn_simt_kernel<T, 128>), grid, dim3(64), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Key splits: the largest power of two (<= 8) that keeps the workgroup count
// within two per CU (512) and at least 4 key tiles per split.
static int pick_splits(int B, int heads, int n_q, int n_kv) {
  const int wg = ceil_div(n_q, mfma_attn::BQ) * heads * B;
  const int tiles = n_kv / mfma_attn::BKV;
  int s = 1;
  while (s < 8 && wg * s * 2 <= 512 && tiles % (2 * s) == 0 && tiles / (2 * s) >= 4) s *= 2;
  return s;
}

static size_t part_o_bytes(int splits, int B, int n_q, int H) {
  return ((size_t)splits * B * n_q * H * 4 + 255) / 256 * 256;
}

size_t attention_workspace_bytes(int B, int heads, int n_q, int n_kv, int d, int dtype) {
  if (n_q <= 0 || !attention_uses_mfma(d, n_kv, dtype)) return 0;
  const int s = pick_splits(B, heads, n_q, n_kv);
  if (s == 1) return 0;
  return part_o_bytes(s, B, n_q, heads * d) + (size_t)s * B * heads * n_q * sizeof(float2);
}

static bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15) == 0; }

template <int D>
static void launch_mfma(dim3 grid, const AttnParams& p, hipStream_t s) {
  constexpr int lds = mfma_attn::Geo<D>::LDS;
  auto kern = attn_bf16_mfma_kernel<D>;
  static bool attr = [&] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    return true;
  }();
  (void)attr;
  hipLaunchKernelGGL(kern, grid, dim3(256), lds, s, p);
}

hipError_t launch_attention(const AttnParams& p0, int dtype, hipStream_t s) {
  if (p0.n_q <= 0) return hipSuccess;
  AttnParams p = p0;
  p.splits = 1;
  // the MFMA kernel moves 16-byte chunks of Q, K and V^T (8 keys of V^T at a
  // time, all fresh or all stale)
  const bool aligned = p.fresh_begin % 8 == 0 && p.n_fresh % 8 == 0 && aligned16(p.q) &&
                       aligned16(p.kv_stale) && p.stale_bs % 8 == 0 &&
                       (p.n_fresh == 0 || (aligned16(p.kv_fresh) && p.fresh_bs % 8 == 0 &&
                                           p.fresh_n % 8 == 0 && p.fresh_off % 8 == 0));
  if (attention_uses_mfma(p.d, p.n_kv, dtype) && aligned) {
    const int want = pick_splits(p.B, p.heads, p.n_q, p.n_kv);
    if (want > 1 && p.ws &&
        p.ws_bytes >= attention_workspace_bytes(p.B, p.heads, p.n_q, p.n_kv, p.d, dtype)) {
      p.splits = want;
      p.part_o = reinterpret_cast<float*>(p.ws);
      p.part_ml = reinterpret_cast<float2*>(reinterpret_cast<char*>(p.ws) +
                                            part_o_bytes(want, p.B, p.n_q, p.heads * p.d));
    }
    dim3 grid(ceil_div(p.n_q, mfma_attn::BQ) * p.splits * p.heads * p.B);
    if (p.d == 64)
      launch_mfma<64>(grid, p, s);
    else
      launch_mfma<72>(grid, p, s);
    if (p.splits > 1) {
      const size_t H = (size_t)p.heads * p.d;
      dim3 g2(ceil_div((int)H, 256), p.B * p.n_q);
      hipLaunchKernelGGL(attn_combine_kernel, g2, dim3(256), 0, s, p);
    }
    return hipGetLastError();
  }
  if (dtype == kBF16) return launch_simt<bf16>(p, s);
  return launch_simt<float>(p, s);
}

}  // namespace orch
