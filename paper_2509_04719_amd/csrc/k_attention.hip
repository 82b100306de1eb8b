// Attention of a band's queries over the keys/values of the whole image,
// fresh for the band's tokens and stale (from the buffer) for all others
// (patch parallelism with stale activations, §II-B; Algorithm 1).
//
// bf16 path: a flash-style kernel on v_mfma_f32_32x32x16_bf16.  Each
// workgroup owns 128 queries of one (branch, head); each wave 32 of them.
// Scores are formed transposed, S^T = K Q^T, so that a lane owns one query
// column: the running max of the online softmax stays in-lane, and the
// probabilities it holds are directly the B operand of O^T = V^T P^T.
// K tiles ([64 keys][d]) and V^T tiles ([d][64 keys]) are staged through
// double-buffered LDS; the V^T layout of the buffer makes both tile loads
// contiguous 16-byte rows.  In LDS the keys of each 16-key chunk of V^T are
// permuted so that the 8 keys a lane's P fragment covers are contiguous (one
// ds_read_b128), and row strides are chosen for the 64-bank LDS.  When the
// head dimension is padded (d = 72 -> 96 rows of O^T), one padding row of
// V^T holds ones, so the PV product also accumulates the softmax
// denominator.  exp2 runs on v_exp_f32 with log2(e)/sqrt(d) folded into the
// exponent; the running max is raised lazily (only past a 2^8 margin), so
// O is rarely rescaled.  Built with MFMA accumulators in VGPRs, so the
// softmax reads the scores without AGPR copies.
//
// fp32 path (and unsupported shapes): one thread per query, online softmax.
#include "common.h"
#include "kernels.h"

namespace orch {

namespace mfma_attn {
constexpr int BQ = 128, BKV = 64;

template <int D>
struct Geo {
  static constexpr int DP = (D + 15) / 16 * 16;  // QK^T contraction, padded to 16
  static constexpr int NC = DP / 16;
  static constexpr int DV = (D + 31) / 32 * 32;  // rows of O^T, padded to 32
  static constexpr int NT = DV / 32;
  static constexpr bool ONES = DV > D;           // padding row D of V^T holds 1.0
  // LDS strides in bf16: 16 consecutive rows of a 16-byte column hit 16
  // distinct 4-bank groups (row stride = 4 * odd banks)
  static constexpr int KS = ((DP / 2) % 8 == 4) ? DP : DP + 8;
  static constexpr int VS = BKV + 8;
  static constexpr int K_CHUNKS = BKV * (D / 8);
  static constexpr int V_CHUNKS = D * (BKV / 8);
  static constexpr int K_IT = (K_CHUNKS + 255) / 256;
  static constexpr int V_IT = (V_CHUNKS + 255) / 256;
  static constexpr int K_BUF = BKV * KS, V_BUF = DV * VS;
};

// Register staging of one K tile ([64 keys][D]) and one V^T tile ([D][64
// keys]) for 256 threads.  K chunk c: key row c / (D/8), 8-dim chunk c % (D/8).
// V^T chunk c: dim row c / 8, 8-key chunk kc = c % 8; in LDS the 4+4 keys of
// that chunk go to positions (kc/2)*16 + (kc%2)*4 and +8, so that within a
// 16-key group a lane with half h finds keys {4h..4h+3, 8+4h..8+4h+3}
// contiguous.  Idle slots (the tile does not split evenly over 256 threads)
// re-read a valid chunk and skip the store.
template <int D>
struct Stage {
  using G = Geo<D>;
  int k_row[G::K_IT], k_col[G::K_IT], k_dst[G::K_IT], v_row[G::V_IT], v_kc[G::V_IT],
      v_dst[G::V_IT], k_on[G::K_IT], v_on[G::V_IT];
  uint4 rk[G::K_IT], rv[G::V_IT];

  __device__ __forceinline__ void init(int tid) {
#pragma unroll
    for (int i = 0; i < G::K_IT; ++i) {
      const int c = tid + 256 * i;
      k_on[i] = c < G::K_CHUNKS;
      k_row[i] = k_on[i] ? c / (D / 8) : 0;
      k_col[i] = k_on[i] ? (c % (D / 8)) * 8 : 0;
      k_dst[i] = k_row[i] * G::KS + k_col[i];
    }
#pragma unroll
    for (int i = 0; i < G::V_IT; ++i) {
      const int c = tid + 256 * i;
      v_on[i] = c < G::V_CHUNKS;
      v_row[i] = v_on[i] ? c >> 3 : 0;
      v_kc[i] = v_on[i] ? c & 7 : 0;
      v_dst[i] = v_row[i] * G::VS + (v_kc[i] >> 1) * 16 + (v_kc[i] & 1) * 4;
    }
  }
  __device__ __forceinline__ void load_k(int n0, const AttnParams& p, const bf16* kf,
                                         const bf16* ks) {
#pragma unroll
    for (int i = 0; i < G::K_IT; ++i) {
      const int n = n0 + k_row[i];
      const int f = n - p.fresh_begin;
      const bf16* src = ((unsigned)f < (unsigned)p.n_fresh) ? kf + (size_t)f * D : ks + (size_t)n * D;
      rk[i] = *reinterpret_cast<const uint4*>(src + k_col[i]);
    }
  }
  __device__ __forceinline__ void load_v(int n0, const AttnParams& p, const bf16* vf,
                                         const bf16* vs) {
#pragma unroll
    for (int i = 0; i < G::V_IT; ++i) {
      const int n = n0 + v_kc[i] * 8;
      const int f = n - p.fresh_begin;
      const bf16* src = ((unsigned)f < (unsigned)p.n_fresh)
                            ? vf + (size_t)v_row[i] * p.n_fresh + f
                            : vs + (size_t)v_row[i] * p.n_kv + n;
      rv[i] = *reinterpret_cast<const uint4*>(src);
    }
  }
  __device__ __forceinline__ void store_k(bf16* sk) const {
#pragma unroll
    for (int i = 0; i < G::K_IT; ++i)
      if (k_on[i]) *reinterpret_cast<uint4*>(sk + k_dst[i]) = rk[i];
  }
  __device__ __forceinline__ void store_v(bf16* sv) const {
#pragma unroll
    for (int i = 0; i < G::V_IT; ++i)
      if (v_on[i]) {
        *reinterpret_cast<uint2*>(sv + v_dst[i]) = make_uint2(rv[i].x, rv[i].y);
        *reinterpret_cast<uint2*>(sv + v_dst[i] + 8) = make_uint2(rv[i].z, rv[i].w);
      }
  }
};

// S^T of one 64-key tile: keys [32 sub, +32) x a wave's 32 queries.  `sk`
// points at this lane's row / half of the K tile in LDS.
struct Scores {
  f32x16 v[2];
};

template <int D>
__device__ __forceinline__ Scores qk_scores(const bf16* sk, const bf16x8 (&qf)[Geo<D>::NC]) {
  Scores sc;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
    for (int r = 0; r < 16; ++r) sc.v[sub][r] = 0.0f;
#pragma unroll
    for (int c = 0; c < Geo<D>::NC; ++c) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(sk + sub * 32 * Geo<D>::KS + c * 16);
      sc.v[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[c], sc.v[sub], 0, 0, 0);
    }
  }
  return sc;
}

}  // namespace mfma_attn

template <int D>
__global__ __launch_bounds__(256) void attn_bf16_mfma_kernel(AttnParams p) {
  using namespace mfma_attn;
  using G = Geo<D>;
  constexpr int NC = G::NC, NT = G::NT, DV = G::DV, KS = G::KS, VS = G::VS;
  constexpr int K_IT = G::K_IT, V_IT = G::V_IT;
  static_assert(((KS / 2) % 4 == 0) && (((KS / 2) / 4) % 2 == 1), "K stride");

  __shared__ __attribute__((aligned(16))) bf16 sK[2][G::K_BUF];
  __shared__ __attribute__((aligned(16))) bf16 sV[2][G::V_BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int lc = lane & 31;
  const int b = blockIdx.z;
  const int head = blockIdx.y;
  const int n_qt = (p.n_q + BQ - 1) / BQ;
  const int split = blockIdx.x / n_qt;            // key split of this workgroup
  const int q0 = (blockIdx.x - split * n_qt) * BQ;
  const int H = p.heads * D;
  const int kv_len = p.n_kv / p.splits;           // multiple of BKV (launcher)
  const int kv0 = split * kv_len;

  const bf16* qbase = reinterpret_cast<const bf16*>(p.q) + ((size_t)b * p.heads + head) * p.n_q * D;
  const bf16* ks = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)head * p.n_kv * D;
  const bf16* vs = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)p.n_kv * H + (size_t)head * D * p.n_kv;
  const bf16* kf = ks;
  const bf16* vf = vs;
  if (p.n_fresh > 0) {
    kf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)head * p.n_fresh * D;
    vf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.n_fresh * H +
         (size_t)head * D * p.n_fresh;
  }

  // padding: K columns [D, KS) are zero; V^T rows [D, DV) are zero except
  // row D, which is one when present (never overwritten by tile loads)
  for (int i = tid; i < 2 * BKV * (KS - D); i += 256) {
    const int buf = i / (BKV * (KS - D));
    const int rem = i - buf * BKV * (KS - D);
    sK[buf][(rem / (KS - D)) * KS + D + rem % (KS - D)] = (bf16)0.0f;
  }
  if constexpr (DV > D) {
    for (int i = tid; i < 2 * (DV - D) * VS; i += 256) {
      const int buf = i / ((DV - D) * VS);
      const int rem = i - buf * (DV - D) * VS;
      sV[buf][D * VS + rem] = (bf16)(rem < VS ? 1.0f : 0.0f);
    }
  }

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

  Stage<D> stg;
  stg.init(tid);
  const float scale = 1.4426950408889634f / sqrtf((float)D);  // log2(e) / sqrt(d)
  float m_run = -1e30f, l_run = 0.0f;
  f32x16 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;

  const int k_rd = lc * KS + h * 8;   // + sub*32*KS + c*16
  const int v_rd = lc * VS + h * 8;   // + t*32*VS + c*16

  // Key tiles: K and V^T of tile it in sK / sV[it & 1]; the next tile is
  // loaded into registers during this one and stored before the barrier.
  // The loads are unconditional (past the end they re-read the last tile,
  // which is then not stored) so the staging stays in registers.
  const int NIT = kv_len / BKV;
  stg.load_k(kv0, p, kf, ks);
  stg.load_v(kv0, p, vf, vs);
  stg.store_k(sK[0]);
  stg.store_v(sV[0]);
  __syncthreads();

  for (int it = 0; it < NIT; ++it) {
    const int buf = it & 1;
    stg.load_k(kv0 + min(it + 1, NIT - 1) * BKV, p, kf, ks);
    stg.load_v(kv0 + min(it + 1, NIT - 1) * BKV, p, vf, vs);
    const Scores sc = qk_scores<D>(sK[buf] + k_rd, qf);

    // online softmax over this lane's query column.  The running max is only
    // raised when some lane's tile max exceeds it by more than 8 (log2
    // units): until then exp2(s - m_run) <= 2^8, exact in fp32 and in range
    // for bf16, and O and the denominator keep a common scale, so O is
    // rarely rescaled.
    float mx = fmaxf(sc.v[0][0], sc.v[1][0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(sc.v[0][r], sc.v[1][r]));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave)) * scale;
    float alpha = 1.0f;
    if (__any(mx > m_run + 8.0f)) {
      const float m_new = fmaxf(m_run, mx);
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
    }
    float psum = 0.0f;
    bf16x8 pf[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int sub = c >> 1;
      const int g0 = 2 * (c & 1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = 4 * (g0 + (e >> 2)) + (e & 3);
        const float pv = __builtin_amdgcn_exp2f(fmaf(sc.v[sub][r], scale, -m_run));
        if constexpr (!G::ONES) psum += pv;
        pf[c][e] = (bf16)pv;
      }
    }
    if constexpr (!G::ONES) l_run = l_run * alpha + psum;

    // O^T += V^T P^T
    const bf16* sv = sV[buf];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(sv + v_rd + t * 32 * VS + c * 16);
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[c], o[t], 0, 0, 0);
      }
    }
    if (it + 1 < NIT) {
      stg.store_k(sK[buf ^ 1]);
      stg.store_v(sV[buf ^ 1]);
    }
    __syncthreads();
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
    kf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)head * p.n_fresh * D;
    vf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.n_fresh * H +
         (size_t)head * D * p.n_fresh;
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
      const float v = fresh ? to_f<T>(vf[(size_t)d * p.n_fresh + f]) : to_f<T>(vs[(size_t)d * p.n_kv + n]);
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

hipError_t launch_attention(const AttnParams& p0, int dtype, hipStream_t s) {
  if (p0.n_q <= 0) return hipSuccess;
  AttnParams p = p0;
  p.splits = 1;
  const bool aligned = (p.fresh_begin % 8 == 0) && (p.n_fresh % 8 == 0);
  if (attention_uses_mfma(p.d, p.n_kv, dtype) && aligned) {
    const int want = pick_splits(p.B, p.heads, p.n_q, p.n_kv);
    if (want > 1 && p.ws &&
        p.ws_bytes >= attention_workspace_bytes(p.B, p.heads, p.n_q, p.n_kv, p.d, dtype)) {
      p.splits = want;
      p.part_o = reinterpret_cast<float*>(p.ws);
      p.part_ml = reinterpret_cast<float2*>(reinterpret_cast<char*>(p.ws) +
                                            part_o_bytes(want, p.B, p.n_q, p.heads * p.d));
    }
    dim3 grid(ceil_div(p.n_q, mfma_attn::BQ) * p.splits, p.heads, p.B);
    if (p.d == 64)
      hipLaunchKernelGGL(attn_bf16_mfma_kernel<64>, grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL(attn_bf16_mfma_kernel<72>, grid, dim3(256), 0, s, p);
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
