// Graph-specialised kernels: HIP source generated for one loaded graph and compiled at run time
// with hiprtc for gfx950.
//
// A loaded graph is immutable and is evaluated for millions of candidates, so the library
// writes the forward pass (Eq. 1-3, one step per candidate-dependent node in a topological
// order), the backward slack pass and the selection epilogue out as straight-line code for that
// graph.  Every finish time is then a named value the compiler keeps in a VGPR, every pack's
// table row offset is an LDS immediate, the level byte of pack p is extracted with a constant
// shift (one SDWA shift-left selects the byte and scales it to the table stride), and there is
// no per-node scalar decoding.  The arithmetic is exactly that of the interpreted kernels: the
// same fp32 maxima and additions, energies summed in fp32 blocks of 64 packs (in the same
// order) added into fp64, so both paths give bit-identical results.
#include <hip/hip_runtime_api.h>
#include <hip/hiprtc.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <sstream>
#include <string>
#include <vector>

#include "emo_internal.h"
#include "emo_select_src.inc"   // kEmoSelectSource: text of emo_select.h

namespace emo {
namespace {

std::string flit(float x) {
    // exact hexadecimal float literal
    char buf[64];
    if (x == 0.f) return "0.0f";
    std::snprintf(buf, sizeof(buf), "%af", static_cast<double>(x));
    return buf;
}

const char *comp(int k) {
    static const char *c[4] = {"x", "y", "z", "w"};
    return c[k];
}

// Level-byte access plan for one graph.  Level words are read straight from the candidate's
// row (16- or 4-byte loads), a fixed distance ahead of their first use.  Each chunk's words
// pass through an empty volatile asm at the point where the chunk's packs start: the table
// reads that depend on them cannot be hoisted above it, and the row pointer passes through one
// before every prefetch, so the scheduler cannot pull every load of a long row to the top of
// the kernel (which would need two VGPRs per pack and spill).
//
// Invalid levels: with F a power of two, a level byte is used as is wherever p*F + 255 stays
// inside the table (one SDWA shift selects and scales it) and masked to [0, F) near the end of
// the table; bits outside the masks record an invalid level.  Otherwise the table carries
// kTablePad spare entries and a SIMD-within-a-register test flags bytes >= F.
struct LevelPlan {
    int P, F;
    int width;            // 16: uint4 words, 4: u32 words, 1: bytes
    bool pow2;
    std::string pfx = "L";        // name prefix of the level words
    bool checks = true;           // record invalid level bytes in `bad`
    long long base_pack = 0;      // pack whose table row starts at entry 0 of `tab`
    long long tab_end = 0;        // table entries readable from entry 0
    std::vector<char> loaded, released;
    std::ostringstream *o;
    // Level words are loaded a whole 128-byte line of the row at a time (all of a group's
    // loads back to back, so the line is fetched from L2 once) and one group ahead of use.
    static constexpr int kGroupBytes = 128;

    int group_words() const { return kGroupBytes / width; }

    unsigned fmask() const { return static_cast<unsigned>(F - 1) * 0x01010101u; }
    int nwords() const { return (P + width - 1) / width; }

    void check(const std::string &w) {
        if (F >= 256 || !checks) return;
        if (pow2) {
            *o << "  bad |= " << w << ";\n";
        } else if (F <= 128) {
            unsigned c = static_cast<unsigned>(0x80 - F) * 0x01010101u;
            *o << "  bad |= ((" << w << " & 0x7f7f7f7fu) + 0x" << std::hex << c << std::dec
               << "u) | " << w << ";\n";
        } else {
            for (int k = 0; k < 4; ++k)
                *o << "  bad |= (((" << w << " >> " << 8 * k << ") & 0xffu) >= " << F
                   << "u) ? 0x80u : 0u;\n";
        }
    }

    // declare_row: declare `rowp` (the row as words); preload: load the first group now.
    void begin(bool declare_row = true, bool preload = true) {
        if (declare_row) *o << row_decl(width);
        loaded.assign(nwords() + 1, 0);
        released.assign(nwords() + 1, 0);
        if (width == 1 || !preload) return;
        load_group(0);
    }

    static std::string row_decl(int width) {
        // global address space: the pointer keeps it through the empty asm statements that
        // order the loads (a generic pointer there would turn them into flat loads, which also
        // count against the LDS wait counter)
        if (width == 16) return "  const EMO_GLOBAL emo_u32x4 *rowp = (const EMO_GLOBAL emo_u32x4 *)row;\n";
        if (width == 4) return "  const EMO_GLOBAL unsigned int *rowp = (const EMO_GLOBAL unsigned int *)row;\n";
        return "  const EMO_GLOBAL u8 *rowb = (const EMO_GLOBAL u8 *)row;\n";
    }

    void load(int q) {
        if (q >= nwords() || loaded[q]) return;
        loaded[q] = 1;
        *o << "  " << (width == 16 ? "emo_u32x4" : "unsigned int") << " " << pfx << q << " = rowp[" << q << "];\n";
    }

    void load_group(int gidx) {
        for (int q = gidx * group_words(); q < (gidx + 1) * group_words(); ++q) load(q);
    }

    // Byte loads (width 1) are released kByteBatch at a time.
    static constexpr int kByteBatch = 16;
    int bytes_loaded = 0;

    bool needs_release(int p) const {
        if (width == 1) return bytes_loaded % kByteBatch == 0;
        return !released[p / width];
    }

    // Releases chunk q.  `ride` names values computed before this point (the energy partial
    // sum and the finish times still needed later) that pass through the same barrier, so the
    // arithmetic of the previous chunk completes before this chunk's table reads start.
    void release(int q, const std::vector<std::string> &ride) {
        if (width == 1) {   // the next batch of byte loads reads through a new row pointer
            std::vector<std::string> ops = {"rowb"};
            ops.insert(ops.end(), ride.begin(), ride.end());
            for (size_t b = 0; b < ops.size(); b += 24) {
                *o << "  __asm__ __volatile__(\"\" :";
                for (size_t k = b; k < ops.size() && k < b + 24; ++k)
                    *o << (k == b ? " " : ", ") << "\"+v\"(" << ops[k] << ")";
                *o << ");\n";
            }
            return;
        }
        const int gidx = q / group_words();
        if (!loaded[q] || (q % group_words() == 0 && (gidx + 1) * group_words() < nwords() &&
                           !loaded[(gidx + 1) * group_words()])) {
            *o << "  __asm__ __volatile__(\"\" : \"+v\"(rowp));\n";
            load_group(gidx);
            load_group(gidx + 1);
        }
        std::string w = pfx + std::to_string(q);
        std::vector<std::string> ops;
        if (width == 16) {
            ops.push_back(w);
        } else {
            ops.push_back(w);
        }
        ops.insert(ops.end(), ride.begin(), ride.end());
        // inline asm takes at most 30 operands
        for (size_t b = 0; b < ops.size(); b += 24) {
            *o << "  __asm__ __volatile__(\"\" :";
            for (size_t k = b; k < ops.size() && k < b + 24; ++k)
                *o << (k == b ? " " : ", ") << "\"+v\"(" << ops[k] << ")";
            *o << ");\n";
        }
        if (width == 16) {
            for (int k = 0; k < 4; ++k) check(w + "." + comp(k));
        } else {
            check(w);
        }
        released[q] = 1;
    }

    // Passes every loaded word through an empty asm statement, so that later uses of the
    // level bytes are computed again from the words (not kept from earlier uses).
    void launder() {
        if (width == 1) {
            *o << "  __asm__ __volatile__(\"\" : \"+v\"(rowb));\n";
            return;
        }
        std::vector<std::string> ops;
        for (int q = 0; q < nwords(); ++q)
            if (loaded[q] && released[q]) ops.push_back(pfx + std::to_string(q));
        for (size_t b = 0; b < ops.size(); b += 16) {
            *o << "  __asm__ __volatile__(\"\" :";
            for (size_t k = b; k < ops.size() && k < b + 16; ++k)
                *o << (k == b ? " " : ", ") << "\"+v\"(" << ops[k] << ")";
            *o << ");\n";
        }
    }

    // Byte loads only: loads pack p's level byte again (after launder(), which gives the row
    // pointer a new value, so the load is not merged with the first one) and returns its
    // expression.  Keeps the byte out of a register between the two uses.
    std::string reload_byte(int p) {
        const std::string b = pfx + "r" + std::to_string(p);
        *o << "  const unsigned int " << b << " = rowb[" << p << "];\n";
        if (pow2 && F < 256 && !raw_ok(p)) return "(" + b + " & " + std::to_string(F - 1) + "u)";
        return b;
    }

    // Returns the expression of pack p's level byte (emitting loads and checks as needed).
    std::string byte_of(int p) {
        std::ostringstream e;
        if (width == 1) {
            const std::string b = pfx + "b" + std::to_string(p);
            *o << "  const unsigned int " << b << " = rowb[" << p << "];\n";
            ++bytes_loaded;
            if (F < 256 && checks) *o << "  bad |= (" << b << " >= " << F << "u) ? 0x80808080u : 0u;\n";
            if (pow2 && F < 256 && !raw_ok(p)) e << "(" << b << " & " << (F - 1) << "u)";
            else e << b;
            return e.str();
        }
        const int q = p / width;
        std::string w = pfx + std::to_string(q);
        if (width == 16) w += std::string(".") + comp((p % 16) / 4);
        const unsigned m = (pow2 && F < 256 && !raw_ok(p)) ? static_cast<unsigned>(F - 1) : 0xffu;
        e << "((" << w << " >> " << 8 * (p % 4) << ") & " << m << "u)";
        return e.str();
    }

    // Whether any byte value at pack p indexes inside the readable table.
    bool raw_ok(int p) const { return !pow2 || (p - base_pack) * F + 255 < tab_end; }

    // Table entry of pack p's row.
    long long row_entry(int p) const { return (p - base_pack) * F; }

    // Bits of `bad` that mark an invalid level.
    std::string bad_bits() const {
        if (F >= 256) return "0u";
        if (pow2) {
            std::ostringstream e;
            e << "0x" << std::hex << (~fmask()) << std::dec << "u";
            return e.str();
        }
        return "0x80808080u";
    }
};

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

std::string est_expr(const JitGraph &g, int i, const char *prefix) {
    const JitOp &op = g.ops[i];
    std::string e;
    bool have = false;
    for (int k : op.in) {
        std::string v = std::string(prefix) + std::to_string(k);
        e = have ? "fmaxf(" + e + ", " + v + ")" : v;
        have = true;
    }
    // finish times are >= 0, so a zero floor from candidate-independent predecessors only
    // matters for a node without candidate-dependent ones
    if (op.cst != 0.f || !have) e = have ? "fmaxf(" + e + ", " + flit(op.cst) + ")" : flit(op.cst);
    return e;
}

// Options of a forward walk over the steps [a, b).
struct RangeOpts {
    int a = 0, b = 0;
    bool accumulate = true;                        // makespan T and energy (eb, ed) as well
    int npk0 = 0;                                  // pack steps before a (energy block phase)
    const std::vector<int> *ck_row = nullptr;      // store f_i to checkpoint row ck_row[i] >= 0
    const std::vector<char> *ck_always = nullptr;  // the row is read by a later forward kernel
    std::string pfx = "L";
    long long base_pack = 0, tab_end = 0;          // table window (LevelPlan)
    bool declare_row = true, preload = true;
    bool checks = true;                            // record invalid level bytes in `bad`
    bool time_only = false;                        // read times only: tab[..] + tsel
    std::string tsel;                              // "" (times table) or ".x" ((t, e) table)
    const std::vector<char> *ck_copy = nullptr;    // copy f_i to c<i> where set
    int pre_lo = 0, pre_hi = 0;                    // level words pfx<q>, pre_lo <= q < pre_hi,
                                                   // were loaded before the walk
    int blk_row0 = -1;                             // >= 0: store each energy block (64 packs
                                                   // from npk0) to row blk_row0 + q of Ebg
};

// Forward walk over steps [a, b) (Eq. 1): declares f<i> for each of them (values of earlier
// steps must be in scope as f<k>); with accumulate, also updates T, eb, ed and bad, which must
// be declared.  Records the expression of each pack step's level byte in *level_expr.
LevelPlan emit_forward_range(std::ostringstream &o, const JitGraph &g, const RangeOpts &r,
                             std::vector<std::string> *level_expr) {
    LevelPlan lp;
    lp.P = g.P;
    lp.F = g.F;
    lp.width = jit_level_width(g);
    lp.pow2 = is_pow2(g.F);
    lp.pfx = r.pfx;
    lp.base_pack = r.base_pack;
    lp.tab_end = r.tab_end;
    lp.checks = r.checks;
    lp.o = &o;
    lp.begin(r.declare_row, r.preload);
    for (int q = r.pre_lo; q < r.pre_hi; ++q) lp.loaded[q] = 1;
    int npk = r.npk0;
    const int n = static_cast<int>(g.ops.size());
    std::vector<int> last_use(n, -1);
    for (int i = 0; i < n; ++i)
        for (int k : g.ops[i].in) last_use[k] = std::max(last_use[k], i);
    int since = r.a;   // first step not yet passed through a barrier
    for (int i = r.a; i < r.b; ++i) {
        const JitOp &op = g.ops[i];
        if (op.pack >= 0 && lp.needs_release(op.pack)) {
            std::vector<std::string> ride;
            if (r.accumulate) ride = r.blk_row0 >= 0 ? std::vector<std::string>{"eb", "bad"}
                                                     : std::vector<std::string>{"eb", "ed", "bad"};
            else ride = {"bad"};
            for (int j = since; j < i; ++j)
                if (last_use[j] >= i) ride.push_back("f" + std::to_string(j));
            lp.release(op.pack / lp.width, ride);
            since = i;
        }
        if (op.pack >= 0) {
            std::string b = lp.byte_of(op.pack);
            if (level_expr) (*level_expr)[i] = b;
            if (r.time_only) {
                o << "  float f" << i << " = " << est_expr(g, i, "f") << " + tab[" << lp.row_entry(op.pack)
                  << " + " << b << "]" << r.tsel << ";\n";
            } else {
                o << "  const float2 te" << i << " = tab[" << lp.row_entry(op.pack) << " + " << b << "];\n";
                o << "  float f" << i << " = " << est_expr(g, i, "f") << " + te" << i << ".x;\n";
            }
            if (r.accumulate) {
                o << "  eb += te" << i << ".y;\n";
                if (++npk % 64 == 0) {
                    if (r.blk_row0 >= 0)
                        o << "  EMO_AT(Ebg, " << r.blk_row0 + (npk - r.npk0) / 64 - 1 << ") = eb;\n  eb = 0.f;\n";
                    else
                        o << "  ed += (double)eb;\n  eb = 0.f;\n";
                }
            }
        } else {
            o << "  float f" << i << " = " << est_expr(g, i, "f") << " + " << flit(op.dur) << ";\n";
        }
        if (r.accumulate && op.out.empty()) o << "  T = fmaxf(T, f" << i << ");\n";
        if (r.ck_copy && (*r.ck_copy)[i]) o << "  c" << i << " = f" << i << ";\n";
        if (r.ck_row && (*r.ck_row)[i] >= 0) {
            if ((*r.ck_always)[i])
                o << "  EMO_AT(ck, " << (*r.ck_row)[i] << ") = f" << i << ";\n";
            else
                o << "  EMO_CKST(" << (*r.ck_row)[i] << ", f" << i << ");\n";
        }
    }
    return lp;
}

// Completes the energy (Eq. 2: table energies plus static power times makespan) and marks a
// candidate with an invalid level byte: declares E and isbad.  nan_carry: an earlier kernel
// marks an invalid level by a NaN energy partial sum.
void emit_forward_finish(std::ostringstream &o, const JitGraph &g, const LevelPlan &lp,
                         bool nan_carry = false) {
    o << "  ed += (double)eb;\n";
    o << "  float E = (float)(ed + (double)" << flit(g.static_power) << " * (double)T);\n";
    o << "  const bool isbad = (bad & " << lp.bad_bits() << ") != 0u" << (nan_carry ? " || ed != ed" : "")
      << ";\n";
    o << "  if (isbad) { T = __builtin_nanf(\"\"); E = __builtin_nanf(\"\"); }\n";
}

// Forward pass of the whole graph: declares f<i> (finish time) for every step, and T, E, bad,
// isbad; records the expression of each pack step's level byte in *level_expr.
LevelPlan emit_forward(std::ostringstream &o, const JitGraph &g, std::vector<std::string> *level_expr) {
    o << "  unsigned int bad = 0u;\n  float eb = 0.f;\n  double ed = 0.0;\n";
    o << "  float T = " << flit(g.t_const) << ";\n";
    RangeOpts r;
    r.b = static_cast<int>(g.ops.size());
    r.tab_end = static_cast<long long>(g.P) * g.F;
    LevelPlan lp = emit_forward_range(o, g, r, level_expr);
    emit_forward_finish(o, g, lp);
    return lp;
}

// Slack output staging: packs [p0, p0 + kc) of the wave's 64 candidates are collected in LDS
// as stg[pack - p0][lane] (row stride 65 floats, conflict-free writes) and written with 16-byte
// stores; with kc = 32 each candidate's segment is one whole 128-byte line.
int stage_chunk(int P) { return P % 32 == 0 ? 32 : 16; }

// Backward pass for per-pack slack (requires the forward's f<i>, T and the level words).
// Pack durations are read from the table again at an index offset by a zero the compiler cannot
// see through, so the forward's loads are not kept alive for the whole pass (and the reads stay
// LDS reads with immediate offsets).
void emit_backward(std::ostringstream &o, const JitGraph &g, bool staged,
                   const std::vector<std::string> &level_expr) {
    const int n = static_cast<int>(g.ops.size());
    o << "  const float Tb = isbad ? 0.f : T;\n";
    o << "  unsigned int zb = 0u;\n  __asm__ __volatile__(\"\" : \"+v\"(zb));\n";
    for (int i = n - 1; i >= 0; --i) {
        const JitOp &op = g.ops[i];
        std::string lft;
        if (op.out.empty()) {
            lft = "Tb";
        } else {
            bool have = false;
            for (int k : op.out) {
                std::string v = "s" + std::to_string(k);
                lft = have ? "fminf(" + lft + ", " + v + ")" : v;
                have = true;
            }
        }
        o << "  const float lf" << i << " = " << lft << ";\n";
        std::string dur = flit(op.dur);
        if (op.pack >= 0) {
            o << "  const float t" << i << " = tab[zb + " << static_cast<long long>(op.pack) * g.F << " + "
              << level_expr[i] << "].x;\n";
            dur = "t" + std::to_string(i);
        }
        if (!op.in.empty()) o << "  const float s" << i << " = lf" << i << " - " << dur << ";\n";
        if (op.pack >= 0) {
            const int p = op.pack;
            const int kc = stage_chunk(g.P);
            if (staged) {
                o << "  stg[" << (p % kc) * 65 << " + lane] = lf" << i << " - f" << i << ";\n";
                if (p % kc == 0) o << "  emo_flush(stg, stg_bad, S, wbase, B, " << p << ");\n";
            } else {
                o << "  if (active) S[cand * " << g.P << "LL + " << p << "] = isbad ? __builtin_nanf(\"\") : lf"
                  << i << " - f" << i << ";\n";
            }
        }
    }
}

// Device routine that writes the slack of packs [p0, p0 + EMO_KC) of the wave's 64 candidates
// from the LDS staging area (rows of P floats per candidate).
std::string flush_source(int P) {
    return std::string(R"(
// Writes the slack of packs [p0, p0 + EMO_KC) of the wave's 64 candidates, staged in LDS.
__device__ __forceinline__ void emo_flush(float *stg, const unsigned int *stg_bad,
                                          float *__restrict__ S, long long wbase, long long B,
                                          int p0) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int lane = threadIdx.x % EMO_WAVE;
  constexpr int per_row = EMO_KC / 4;          // 16-byte pieces per candidate segment
#pragma unroll
  for (int m = 0; m < per_row; ++m) {
    const int j = lane + EMO_WAVE * m;
    const int r = j / per_row, part = j % per_row;
    float4 v;
    v.x = stg[(4 * part + 0) * 65 + r];
    v.y = stg[(4 * part + 1) * 65 + r];
    v.z = stg[(4 * part + 2) * 65 + r];
    v.w = stg[(4 * part + 3) * 65 + r];
    if (stg_bad[r]) { v.x = EMO_NAN; v.y = EMO_NAN; v.z = EMO_NAN; v.w = EMO_NAN; }
    const long long row = wbase + r;
    if (row < B) *(float4 *)(S + row * )" + std::to_string(P) + R"(LL + p0 + 4 * part) = v;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
)");
}

const char *kPrelude = R"(
typedef unsigned char u8;
#define EMO_AT(buf, r) (*(__typeof__(&(buf)[0]))((const char *)((buf) + (long long)(r) * bp) + o4))
typedef unsigned int emo_u32x4 __attribute__((ext_vector_type(4)));
typedef float emo_f32x4 __attribute__((ext_vector_type(4)));
#define EMO_GLOBAL __attribute__((address_space(1)))
#define EMO_NAN __builtin_nanf("")
)";

}  // namespace

std::string jit_generate(const JitGraph &g, bool with_slack, bool tab_lds, int block) {
    std::ostringstream o;
    o << "#define EMO_BLOCK " << block << "\n" << kPrelude << kEmoSelectSource << "\n";
    const long long ntab = static_cast<long long>(g.P) * g.F + (is_pow2(g.F) ? 0 : kTablePad);
    o << "#define NTAB " << ntab << "\n";
    // table access
    if (tab_lds) {
        o << "#define EMO_TABLE_DECL __shared__ float2 tab[NTAB]; \\\n"
             "  for (int i_ = threadIdx.x; i_ < NTAB; i_ += EMO_BLOCK) tab[i_] = tabg[i_]; \\\n"
             "  __syncthreads();\n";
    } else {
        o << "#define EMO_TABLE_DECL const float2 *__restrict__ tab = tabg;\n";
    }
    // Persistent workgroups: each loads the table once and walks groups of EMO_BLOCK
    // candidates grp = blockIdx.x, blockIdx.x + gridDim.x, ...
    o << "#define EMO_GROUP_LOOP \\\n"
         "  for (long long grp = blockIdx.x; grp * EMO_BLOCK < B; grp += gridDim.x)\n";
    o << "#define EMO_LANE_SETUP \\\n"
         "  const long long gid = grp * EMO_BLOCK + threadIdx.x; \\\n"
         "  const bool active = gid < B; \\\n"
         "  long long cand = active ? gid : B - 1; \\\n"
         "  (void)active;\n";

    // forward function body as a macro-free inline function over (row, tab)
    std::ostringstream fwd;
    emit_forward(fwd, g, nullptr);

    o << "struct EmoFwd { float T; float E; };\n";
    o << "__device__ __forceinline__ EmoFwd emo_forward(const u8 *__restrict__ row, "
         "const float2 *__restrict__ tab) {\n"
      << fwd.str() << "  EmoFwd r; r.T = T; r.E = E; return r;\n}\n";

    // forward pass, optional makespan/energy outputs, feasibility mask and selection partials
    o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
         "emo_sp_select(const u8 *__restrict__ lv, long long B, const float2 *__restrict__ tabg,\n"
         "              float *__restrict__ To, float *__restrict__ Eo,\n"
         "              EmoTargets tg) {\n"
         "  EMO_TABLE_DECL\n  EMO_GROUP_LOOP {\n  EMO_LANE_SETUP\n"
         "  const EmoFwd r = emo_forward(lv + cand * "
      << g.P << "LL, tab);\n"
         "  if (active) { if (To) To[cand] = r.T; if (Eo) Eo[cand] = r.E; }\n"
         "  if (tg.n) emo_select_all(grp, active, r.T, r.E, cand, B, tg);\n"
         "  }\n}\n";

    if (with_slack) {
        const bool staged = g.pack_monotone && g.P % 16 == 0;
        if (staged) {
            const int kc = stage_chunk(g.P);
            o << "#define EMO_KC " << kc << "\n";
            o << flush_source(g.P);
        }
        o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
             "emo_sp_slack(const u8 *__restrict__ lv, long long B, const float2 *__restrict__ tabg,\n"
             "             float *__restrict__ S, float *__restrict__ To, float *__restrict__ Eo,\n"
             "             EmoTargets tg) {\n"
             "  EMO_TABLE_DECL\n"
             "  const int lane = threadIdx.x % EMO_WAVE;\n"
             "  const int wave = threadIdx.x / EMO_WAVE;\n"
             "  (void)lane;\n";
        if (staged) {
            o << "  __shared__ float stg_all[EMO_WAVES_PER_BLOCK][EMO_KC * 65];\n"
                 "  __shared__ unsigned int bad_all[EMO_WAVES_PER_BLOCK][EMO_WAVE];\n"
                 "  float *stg = stg_all[wave];\n"
                 "  unsigned int *stg_bad = bad_all[wave];\n";
        }
        o << "  EMO_GROUP_LOOP {\n  EMO_LANE_SETUP\n"
             "  const long long wbase = grp * EMO_BLOCK + wave * EMO_WAVE;\n"
             "  (void)wbase;\n";
        o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
        std::vector<std::string> level_expr(g.ops.size());
        LevelPlan lp = emit_forward(o, g, &level_expr);
        o << "  if (active) { if (To) To[cand] = T; if (Eo) Eo[cand] = E; }\n";
        if (staged) o << "  stg_bad[lane] = isbad ? 1u : 0u;\n";
        lp.launder();
        emit_backward(o, g, staged, level_expr);
        o << "  if (tg.n) emo_select_all(grp, active, T, E, cand, B, tg);\n";
        o << "  }\n}\n";
    }
    return o.str();
}

// ------------------------------------------------------------------ time-interval kernels
//
// Time-interval policies (the policy form of Sec. IV-A as Alg. 1 evaluates it): a candidate's
// row holds one level per interval [T_i, T_{i+1}) of the batch's change points, and a pack runs
// at the level of the interval that holds its start time.  The forward pass is the same
// straight-line code as emo_sp_select; before each pack's table read, its interval comes from a
// bucket table built in LDS from the change points: with u(x) = fl(x * scale), bucket
// b = floor(min(u(est), M - 1)) holds the count of change points whose bucket is below b and the
// one point whose bucket is b (+inf if none; the host picks scale so that no two points share a
// bucket).  Since fl(x * scale) is monotone in x, every point of a lower bucket is <= est, every
// point of a higher one is > est, and the one in bucket b is compared directly: the count of
// points <= est is exact, as in the interpreting kernel.  Energies and the idle term follow the
// interpreting kernel's order, so both give bit-identical results.

std::string jit_generate_intervals(const JitGraph &g, bool tab_lds, int block) {
    std::ostringstream o;
    o << "#define EMO_BLOCK " << block << "\n" << kPrelude << kEmoSelectSource << "\n";
    const long long ntab = static_cast<long long>(g.P) * g.F;
    o << "#define NTAB " << (ntab > 0 ? ntab : 1) << "\n";
    o << "#define EMO_F " << g.F << "\n";
    o << "struct EmoIvArgs { int K; int M; float scale; int pad; float pts[" << kMaxIntervals - 1
      << "]; float idle[" << kMaxLevels << "]; };\n";
    // a level byte is invalid when it is >= F: SWAR test of the four bytes of a word
    std::string bad_word;
    if (g.F >= 256) {
        bad_word = "0u";
    } else if (g.F <= 128) {
        bad_word = "(((w & 0x7f7f7f7fu) + " + std::to_string((128u - g.F) * 0x01010101u) +
                   "u) | w) & 0x80808080u";
    } else {
        bad_word = "(((w & 0x7f7f7f7fu) + " + std::to_string((256u - g.F) * 0x01010101u) +
                   "u) & w) & 0x80808080u";
    }
    o << R"(
// interval of start time `est`: the number of change points <= est
__device__ __forceinline__ unsigned int emo_interval(float est, const int2 *bk, float scale, int M) {
  const int b = (int)fminf(est * scale, (float)(M - 1));
  const int2 e = bk[b];
  return (unsigned int)e.x + (est >= __int_as_float(e.y) ? 1u : 0u);
}
struct EmoFwd { float T; float E; bool bad; };
)";
    // forward body; the lane's row of K level bytes is in LDS at `myrow` (word aligned)
    o << "__device__ __forceinline__ EmoFwd emo_iv_forward(const u8 *myrow, int K,\n"
         "    const float2 *__restrict__ tab, const int2 *bk, float scale, int M, const float *pts,\n"
         "    const double *dur, const float *idle) {\n"
         "  float T = " << flit(g.t_const) << ";\n"
         "  double eacc = 0.0;\n  float eblk = 0.f;\n";
    const int n = static_cast<int>(g.ops.size());
    std::vector<int> last_use(n, -1);
    for (int i = 0; i < n; ++i)
        for (int k : g.ops[i].in) last_use[k] = std::max(last_use[k], i);
    int npk = 0;
    for (int i = 0; i < n; ++i) {
        const JitOp &op = g.ops[i];
        if (i > 0 && i % 4 == 0) {
            // the finish times still needed and the running sums pass through an empty asm: the
            // scheduler cannot interleave far-apart steps (which would keep many values live)
            std::vector<std::string> live = {"eblk", "T"};
            for (int j = 0; j < i; ++j)
                if (last_use[j] >= i) live.push_back("f" + std::to_string(j));
            for (size_t b = 0; b < live.size(); b += 24) {
                o << "  __asm__ __volatile__(\"\" :";
                for (size_t k = b; k < live.size() && k < b + 24; ++k)
                    o << (k == b ? " " : ", ") << "\"+v\"(" << live[k] << ")";
                o << ");\n";
            }
        }
        o << "  const float e" << i << " = " << est_expr(g, i, "f") << ";\n";
        if (op.pack >= 0) {
            o << "  const unsigned int v" << i << " = emo_interval(e" << i << ", bk, scale, M);\n"
              << "  unsigned int l" << i << " = myrow[v" << i << "];\n"
              << "  l" << i << " = l" << i << " < EMO_F ? l" << i << " : 0u;\n"
              << "  const float2 te" << i << " = tab[" << static_cast<long long>(op.pack) * g.F << " + l" << i
              << "];\n"
              << "  float f" << i << " = e" << i << " + te" << i << ".x;\n"
              << "  eblk += te" << i << ".y;\n";
            if (++npk % kEnergyBlock == 0) o << "  eacc += (double)eblk;\n  eblk = 0.f;\n";
        } else {
            o << "  float f" << i << " = e" << i << " + " << flit(op.dur) << ";\n";
        }
        if (op.out.empty()) o << "  T = fmaxf(T, f" << i << ");\n";
    }
    o << "  eacc += (double)eblk;\n"
         "  // invalid levels anywhere in the row, four bytes a word\n"
         "  const unsigned int *mw = (const unsigned int *)myrow;\n"
         "  unsigned int bad = 0u;\n"
         "  for (int j = 0; 4 * j < K; ++j) {\n"
         "    unsigned int w = mw[j];\n"
         "    if (4 * j + 4 > K) w &= 0xffffffffu >> (8 * (4 * j + 4 - K));   // bytes past the row\n"
         "    bad |= " << bad_word << ";\n"
         "  }\n";
    o << R"(  // idle energy, interval by interval in increasing order: the whole length of the nf
  // intervals that end at or before T (nf: the number of change points <= T, the interval of T),
  // then the part of interval nf below T.  Levels >= F read zeros (their row gives NaN anyway).
  const int nf = (int)emo_interval(T, bk, scale, M);
  for (int j = 0; 4 * j < nf; ++j) {
    const unsigned int w = mw[j];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (4 * j + q < nf) eacc = fma((double)idle[(w >> (8 * q)) & 255u], dur[4 * j + q], eacc);
  }
  const double Td = (double)T;
  const double lo = nf > 0 ? (double)pts[nf - 1] : 0.0;
  if (Td > lo) eacc = fma((double)idle[myrow[nf]], Td - lo, eacc);
  EmoFwd r;
  r.T = T;
  r.E = (float)eacc;
  r.bad = bad != 0u;
  if (r.bad) { r.T = EMO_NAN; r.E = EMO_NAN; }
  return r;
}
)";
    o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
         "emo_iv(const u8 *__restrict__ lv, long long B, const float2 *__restrict__ tabg, EmoIvArgs a,\n"
         "    int copy, float inv_k, float *__restrict__ To, float *__restrict__ Eo, EmoTargets tg) {\n";
    if (tab_lds)
        o << "  __shared__ float2 tab[NTAB];\n"
             "  for (int i_ = threadIdx.x; i_ < NTAB; i_ += EMO_BLOCK) tab[i_] = tabg[i_];\n";
    else
        o << "  const float2 *__restrict__ tab = tabg;\n";
    o << R"(  __shared__ float s_pts[256];
  __shared__ double s_dur[256];      // interval lengths T_{i+1} - T_i (T_0 = 0)
  __shared__ float s_idle[256];      // zero past F
  // dynamic: the bucket table (M entries), then the group's rows, SD words a row
  extern __shared__ __align__(16) unsigned int emo_dyn[];
  const int K = a.K, M = a.M;
  const int SD = ((K + 3) >> 2) | 1;        // odd: a word column of the rows is conflict free
  int2 *s_bk = (int2 *)emo_dyn;
  unsigned int *s_rows = emo_dyn + 2 * M;
  const float scale = a.scale;
  for (int i = threadIdx.x; i < K - 1; i += EMO_BLOCK) s_pts[i] = a.pts[i];
  for (int i = threadIdx.x; i < K - 1; i += EMO_BLOCK)
    s_dur[i] = (double)a.pts[i] - (i > 0 ? (double)a.pts[i - 1] : 0.0);
  for (int i = threadIdx.x; i < 256; i += EMO_BLOCK) s_idle[i] = i < EMO_F ? a.idle[i] : 0.f;
  __syncthreads();
  // bucket b: the number of points whose bucket is below b (they are increasing, and so are
  // their buckets), and the point whose bucket is b, if any
  for (int b = threadIdx.x; b < M; b += EMO_BLOCK) {
    int lo = 0, hi = K - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((int)(s_pts[mid] * scale) < b) lo = mid + 1; else hi = mid;
    }
    const float c = lo < K - 1 && (int)(s_pts[lo] * scale) == b ? s_pts[lo] : __builtin_inff();
    s_bk[b] = make_int2(lo, __float_as_int(c));
  }
  const u8 *my = (const u8 *)(s_rows + threadIdx.x * SD);
  for (long long grp = blockIdx.x; grp * EMO_BLOCK < B; grp += gridDim.x) {
    // the group's rows are contiguous: copy them to LDS with coalesced loads of `copy` bytes
    // (16 when K is a multiple of 16, 4 when of 4, else 1; the batch aligned to match).  Row of
    // byte x: floor((x + 0.5) / K), exact from the fp32 product for x < 2^16, K <= 256.
    __syncthreads();   // the previous group's rows are read (and the tables built)
    {
      const long long r0 = grp * EMO_BLOCK;
      const int nb = (int)(B - r0 < EMO_BLOCK ? B - r0 : EMO_BLOCK) * K;
      const u8 *src = lv + r0 * K;
      if (copy == 16) {
        for (int q = threadIdx.x; q < (nb >> 4); q += EMO_BLOCK) {
          const emo_u32x4 w = ((const emo_u32x4 *)src)[q];
          const int r = (int)(((float)(q << 4) + 0.5f) * inv_k);
          unsigned int *d = s_rows + r * SD + (((q << 4) - r * K) >> 2);
          d[0] = w.x; d[1] = w.y; d[2] = w.z; d[3] = w.w;
        }
      } else if (copy == 4) {
        for (int q = threadIdx.x; q < (nb >> 2); q += EMO_BLOCK) {
          const unsigned int w = ((const unsigned int *)src)[q];
          const int r = (int)(((float)(q << 2) + 0.5f) * inv_k);
          s_rows[r * SD + (((q << 2) - r * K) >> 2)] = w;
        }
      } else {
        for (int q = threadIdx.x; q < nb; q += EMO_BLOCK) {
          const int r = (int)(((float)q + 0.5f) * inv_k);
          ((u8 *)s_rows)[((r * SD) << 2) + q - r * K] = src[q];
        }
      }
    }
    __syncthreads();
    const long long gid = grp * EMO_BLOCK + threadIdx.x;
    const bool active = gid < B;
    const long long cand = active ? gid : B - 1;
    const EmoFwd r = emo_iv_forward(my, K, tab, s_bk, scale, M, s_pts, s_dur, s_idle);
    if (active) { if (To) To[cand] = r.T; if (Eo) Eo[cand] = r.E; }
    if (tg.n) emo_select_all(grp, active, r.T, r.E, cand, B, tg);
  }
}
)";
    return o.str();
}

// ------------------------------------------------------------------ segmented kernels

namespace {
constexpr int kChainSegPacks = 256;        // packs per segment kernel at most (table window)
}  // namespace

ChainPlan jit_chain_plan(const JitGraph &g, bool with_slack, int seg_ops, int sub_ops) {
    ChainPlan cp;
    cp.slack = with_slack;
    const int n = static_cast<int>(g.ops.size());
    std::vector<int> npk_before(n + 1, 0);
    for (int i = 0; i < n; ++i) npk_before[i + 1] = npk_before[i] + (g.ops[i].pack >= 0 ? 1 : 0);
    // Segments end where the pack steps so far are a multiple of 64 (energy blocks and slack
    // chunks never straddle two kernels), after seg_ops steps or kChainSegPacks packs (the
    // table window of a kernel); a short tail joins the last segment when the packs allow.
    cp.seg.push_back(0);
    for (int i = 0, start = 0; i + 1 < n; ++i) {
        const int c = i + 1;
        if (npk_before[c] % 64 != 0) continue;
        const int packs = npk_before[c] - npk_before[start];
        if (c - start < seg_ops && packs < kChainSegPacks) continue;
        const int rest_ops = n - c, rest_packs = npk_before[n] - npk_before[c];
        if (rest_ops < seg_ops / 4 && packs + rest_packs <= kChainSegPacks) continue;
        cp.seg.push_back(c);
        start = c;
    }
    cp.seg.push_back(n);
    std::vector<int> seg_of(n), sub_of(n);
    for (int j = 0; j + 1 < static_cast<int>(cp.seg.size()); ++j) {
        // sub-segments of at least sub_ops steps, cut where the pack steps so far are a multiple
        // of 32, so that a 32-pack slack chunk never waits across two of them
        const int a = cp.seg[j], b = cp.seg[j + 1];
        cp.sub.push_back(a);
        for (int c = a + 1, start = a; c < b; ++c)
            if (c - start >= sub_ops && npk_before[c] % 32 == 0) {
                cp.sub.push_back(c);
                start = c;
            }
        for (int i = a; i < b; ++i) seg_of[i] = j;
    }
    cp.sub.push_back(n);
    for (int r = 0; r + 1 < static_cast<int>(cp.sub.size()); ++r)
        for (int i = cp.sub[r]; i < cp.sub[r + 1]; ++i) sub_of[i] = r;
    cp.ck_row.assign(n, -1);
    cp.ck_always.assign(n, 0);
    cp.bk_row.assign(n, -1);
    for (int i = 0; i < n; ++i) {
        bool later_seg = false, other_sub = false;
        for (int k : g.ops[i].out) {
            later_seg |= seg_of[k] != seg_of[i];
            other_sub |= sub_of[k] != sub_of[i];
        }
        if (later_seg || (with_slack && other_sub)) {
            cp.ck_row[i] = cp.n_ck++;
            cp.ck_always[i] = later_seg;
        }
        if (with_slack) {
            bool earlier = false;
            for (int k : g.ops[i].in) earlier |= seg_of[k] != seg_of[i];
            if (earlier) cp.bk_row[i] = cp.n_bk++;
        }
    }
    cp.staged = with_slack && g.pack_monotone && g.P % 32 == 0;
    cp.block = 256;
    cp.bblock = 512;
    return cp;
}

namespace {

constexpr size_t kChainLdsForward = 48 * 1024;         // table window budget, forward kernels
constexpr size_t kChainLdsBackward = 16 * 1024;        // times window budget, backward kernels

// Table window of one kernel: the rows of the packs its steps visit, staged in LDS when they
// fit, else the whole table in device memory.
struct TabWindow {
    bool lds = false;
    long long base_pack = 0, entries = 0, tab_end = 0;
};

TabWindow chain_window(const JitGraph &g, int a, int b, size_t budget, size_t entry_bytes) {
    int lo = g.P, hi = -1;
    for (int i = a; i < b; ++i)
        if (g.ops[i].pack >= 0) {
            lo = std::min(lo, g.ops[i].pack);
            hi = std::max(hi, g.ops[i].pack);
        }
    TabWindow w;
    w.tab_end = static_cast<long long>(g.P) * g.F;
    if (hi < 0) return w;
    const long long rows = static_cast<long long>(hi - lo + 1) * g.F;
    const long long ent = rows + (is_pow2(g.F) ? 0 : kTablePad);
    if (static_cast<size_t>(ent) * entry_bytes > budget) return w;
    w.lds = true;
    w.base_pack = lo;
    w.entries = ent;
    w.tab_end = rows;
    return w;
}

// Copy of `entries` table elements of `elem_bytes` bytes from tabg + base into the LDS array
// tab by `block` threads: every 16-byte piece a thread copies is requested before the first is
// stored, so the copy costs one round trip to the L2 instead of one per piece (a strided loop
// waits for each load before the next).  Needs tabg + base 16-byte aligned (the device tables
// are, from their allocation); otherwise a plain unrolled loop.  No barrier.
std::string table_copy(long long entries, long long base, int elem_bytes, int block) {
    std::ostringstream o;
    const long long bytes = entries * elem_bytes;
    if ((base * elem_bytes) % 16 != 0 || bytes % 16 != 0) {
        o << "  #pragma unroll\n"
             "  for (int i_ = threadIdx.x; i_ < " << entries << "; i_ += " << block << ") tab[i_] = tabg["
          << base << "LL + i_];\n";
        return o.str();
    }
    const long long pieces = bytes / 16;
    const long long rounds = pieces / block, rest = pieces % block;
    o << "  {\n"
         "  const EMO_GLOBAL emo_u32x4 *src_ = (const EMO_GLOBAL emo_u32x4 *)(tabg + " << base << "LL);\n"
         "  emo_u32x4 *dst_ = (emo_u32x4 *)tab;\n";
    for (long long k = 0; k < rounds; ++k)
        o << "  const emo_u32x4 tc" << k << " = src_[threadIdx.x + " << k * block << "];\n";
    if (rest)
        o << "  const emo_u32x4 tcr = threadIdx.x < " << rest << " ? src_[threadIdx.x + " << rounds * block
          << "] : (emo_u32x4)(0u);\n";
    for (long long k = 0; k < rounds; ++k) o << "  dst_[threadIdx.x + " << k * block << "] = tc" << k << ";\n";
    if (rest) o << "  if (threadIdx.x < " << rest << ") dst_[threadIdx.x + " << rounds * block << "] = tcr;\n";
    o << "  }\n";
    return o.str();
}

void emit_table(std::ostringstream &o, const JitGraph &g, const TabWindow &w, const char *type,
                int elem_bytes, int block) {
    if (!w.lds) {
        o << "  const " << type << " *__restrict__ tab = tabg;\n";
        return;
    }
    o << "  __shared__ " << type << " tab[" << w.entries << "];\n"
      << table_copy(w.entries, w.base_pack * g.F, elem_bytes, block) << "  __syncthreads();\n";
}

// Lane setup of a segmented kernel.  Scratch row r is addressed as a uniform base
// (buf + r * bp) plus the lane's 32-bit byte offset o4 (bp * 4 < 2^32), which the compiler
// folds into one load or store with a scalar base.
// Lanes past the batch evaluate the last candidate (cand = B - 1) again and use its scratch
// slot.  Stores of values that depend only on the candidate's levels (checkpoint rows, slack)
// need no branch: those lanes store exactly the owner's values.  Running sums that the next
// kernel reads back and adds to are stored by the owning lane only.
std::string chain_lanes(int block) {
    std::ostringstream o;
    o << "  const unsigned int g32 = blockIdx.x * " << block << "u + threadIdx.x;\n"
         "  const long long gid = g32;\n"
         "  const bool active = gid < B;\n"
         "  const long long cand = active ? gid : B - 1;\n"
         "  const unsigned int o4 = (unsigned int)cand * 4u;\n"
         "  (void)active;\n";
    return o.str();
}

// Steps before `a` whose finish times steps [a, b) read.
std::vector<int> inputs_before(const JitGraph &g, int a, int b) {
    std::vector<int> v;
    for (int i = a; i < b; ++i)
        for (int k : g.ops[i].in)
            if (k < a) v.push_back(k);
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
    return v;
}

// Level words [*lo, *hi) holding the packs of steps [c, d) (empty when there are none).
void sub_words(const JitGraph &g, int c, int d, int width, int *lo, int *hi) {
    *lo = g.P;
    *hi = 0;
    for (int i = c; i < d; ++i)
        if (g.ops[i].pack >= 0) {
            *lo = std::min(*lo, g.ops[i].pack / width);
            *hi = std::max(*hi, g.ops[i].pack / width + 1);
        }
    if (*lo >= *hi) *lo = *hi = 0;
}

void emit_chain_forward(std::ostringstream &o, const JitGraph &g, const ChainPlan &cp, int j) {
    const int a = cp.seg[j], b = cp.seg[j + 1];
    const bool last = j + 1 == cp.segments();
    int npk0 = 0, npk1 = 0;
    for (int i = 0; i < b; ++i)
        if (g.ops[i].pack >= 0) (i < a ? npk0 : npk1)++;
    npk1 += npk0;
    const TabWindow w = chain_window(g, a, b, kChainLdsForward, sizeof(float) * 2);
    o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
      << "emo_cf" << j << "(const u8 *__restrict__ lv, long long B, long long bp,\n"
         "    const float2 *__restrict__ tabg, float *__restrict__ ck, float *__restrict__ Tc,\n"
         "    double *__restrict__ Edc, float *__restrict__ Ebc, int full, float *__restrict__ To,\n"
         "    float *__restrict__ Eo, EmoTargets tg) {\n";
    emit_table(o, g, w, "float2", 8, cp.block);
    o << chain_lanes(cp.block);
    o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
    // checkpoints only the backward kernels read: stored through a buffer resource whose range
    // is empty without slack (the hardware drops those stores), so no branch splits the code
    o << "  unsigned int bad = 0u;\n"
         "  const int ckn = full ? (int)(unsigned int)(bp * 4) : 0;\n"
         "  (void)ckn;\n"
         "#define EMO_CKST(r, v) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), "
         "__builtin_amdgcn_make_buffer_rsrc((void *)(ck + (long long)(r) * bp), (short)0, ckn, 0x00020000), o4, 0, 0)\n";
    if (j == 0) {
        o << "  float T = " << flit(g.t_const) << ";\n  float eb = 0.f;\n  double ed = 0.0;\n";
    } else {
        o << "  float T = Tc[cand];\n  double ed = Edc[cand];\n";
        o << "  float eb = " << (npk0 % 64 ? "Ebc[cand]" : "0.f") << ";\n";
    }
    for (int k : inputs_before(g, a, b))
        o << "  const float f" << k << " = EMO_AT(ck, " << cp.ck_row[k] << ");\n";
    RangeOpts r;
    r.a = a;
    r.b = b;
    r.npk0 = npk0;
    r.ck_row = &cp.ck_row;
    r.ck_always = &cp.ck_always;
    r.base_pack = w.base_pack;
    r.tab_end = w.tab_end;
    r.preload = false;
    LevelPlan lp = emit_forward_range(o, g, r, nullptr);
    if (!last) {
        o << "  if ((bad & " << lp.bad_bits() << ") != 0u) ed = (double)EMO_NAN;\n";
        // the running makespan and energy are read back and added to by the next kernel: only
        // the lane that owns the candidate stores them (a lane past the batch repeats candidate
        // B - 1 in another wave that may run after its owner's store, and would add twice)
        o << "  if (active) {\n    Tc[cand] = T;\n    Edc[cand] = ed;\n";
        if (npk1 % 64) o << "    Ebc[cand] = eb;\n";
        o << "  }\n";
    } else {
        emit_forward_finish(o, g, lp, j > 0);
        o << "  if (active) Tc[cand] = T;\n"
             "  if (active) { if (To) To[cand] = T; if (Eo) Eo[cand] = E; }\n"
             "  if (tg.n) emo_select_all(blockIdx.x, active, T, E, cand, B, tg);\n";
    }
    o << "}\n\n";
}

// Slack staging of the backward kernels: the slack of packs [p0, p0 + 32) of the wave's 64
// candidates is collected in LDS as an unpadded 32 x 64 tile (8 KB), element (k, r) at
// k * 64 + (r ^ (8 * (k / 4))), then written with 16-byte stores in which 8 lanes cover one
// candidate's 128-byte line.  The XOR keeps both sides free of bank conflicts: a lane writes
// its column (k fixed), and a read of piece b (packs 4b..4b+3) by 64 lanes touches 8 rows
// r = 8m..8m+7 of 8 different swizzles.  Values of a bad candidate are already NaN.
std::string chain_flush_source(int P) {
    std::ostringstream o;
    o << R"(
__device__ __forceinline__ void emo_cflush(const float *stg, float *__restrict__ S,
                                           long long wbase, long long B, int p0) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int lane = threadIdx.x % EMO_WAVE;
  const int b = lane % 8;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const int r = 8 * m + lane / 8;
    const int sw = r ^ (8 * b);
    emo_f32x4 v;
    v.x = stg[(4 * b + 0) * 64 + sw];
    v.y = stg[(4 * b + 1) * 64 + sw];
    v.z = stg[(4 * b + 2) * 64 + sw];
    v.w = stg[(4 * b + 3) * 64 + sw];
    long long row = wbase + r;
    row = row < B ? row : B - 1;   // lanes past the batch hold candidate B - 1's values
    // streaming store: slack is never read back here, and leaving it out of L2 keeps the
    // checkpoint rows that the backward kernels read several times there
    __builtin_nontemporal_store(v, (emo_f32x4 *)(S + row * )" << P << R"(LL + p0 + 4 * b));
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
)";
    return o.str();
}

void emit_chain_backward(std::ostringstream &o, const JitGraph &g, const ChainPlan &cp, int j) {
    const int a = cp.seg[j], b = cp.seg[j + 1];
    const TabWindow w = chain_window(g, a, b, kChainLdsBackward, sizeof(float));
    // 4 waves per SIMD: two workgroups of 8 waves share a CU's LDS (staging + times window)
    o << "extern \"C\" __global__ void __launch_bounds__(" << cp.bblock
      << ") __attribute__((amdgpu_waves_per_eu(4)))\n"
      << "emo_cb" << j << "(const u8 *__restrict__ lv, long long B, long long bp,\n"
         "    const float *__restrict__ tabg, const float *__restrict__ ck,\n"
         "    const float *__restrict__ Tc, float *__restrict__ bk, float *__restrict__ S) {\n";
    if (w.lds) {
        o << "  __shared__ float tab[" << w.entries << "];\n"
          << table_copy(w.entries, w.base_pack * g.F, 4, cp.bblock) << "  __syncthreads();\n";
    } else {
        o << "  const float *__restrict__ tab = tabg;\n";
    }
    o << chain_lanes(cp.bblock);
    o << "  const int lane = threadIdx.x % EMO_WAVE;\n"
         "  const int wave = threadIdx.x / EMO_WAVE;\n"
         "  const long long wbase = (long long)blockIdx.x * " << cp.bblock << " + wave * EMO_WAVE;\n"
         "  (void)lane; (void)wbase;\n";
    if (cp.staged) {
        o << "  __shared__ float stg_all[" << cp.bblock / 64 << "][32 * 64];\n"
             "  float *stg = stg_all[wave];\n";
    }
    o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
    o << "  float *__restrict__ srow = S + cand * " << g.P << "LL;\n  (void)srow;\n";
    o << LevelPlan::row_decl(jit_level_width(g));
    o << "  const float T = Tc[cand];\n  const bool isbad = T != T;\n"
         "  const float Tb = isbad ? 0.f : T;\n";
    o << "  unsigned int zb = 0u;\n  __asm__ __volatile__(\"\" : \"+v\"(zb));\n";
    o << "  unsigned int bad = 0u;\n";
    // latest start times of later segments' steps that this segment's steps precede
    std::vector<int> later;
    for (int i = a; i < b; ++i)
        for (int u : g.ops[i].out)
            if (u >= b) later.push_back(u);
    std::sort(later.begin(), later.end());
    later.erase(std::unique(later.begin(), later.end()), later.end());
    for (int u : later) o << "  const float s" << u << " = EMO_AT(bk, " << cp.bk_row[u] << ");\n";
    for (int i = a; i < b; ++i)
        if (!g.ops[i].in.empty()) o << "  float s" << i << ";\n";
    // sub-segments from last to first: recompute their finish times, then walk them backwards.
    // The checkpoints and level words of the next sub-segment are requested during this one's
    // walk, before its slack stores: on this GPU a wait for a load also waits for every store
    // issued before it, so loads issued after the stores would stall on their completion.
    int r_first = 0;
    while (cp.sub[r_first] < a) ++r_first;
    int r_last = r_first;
    while (cp.sub[r_last + 1] < b) ++r_last;
    const int width = jit_level_width(g);
    for (int r = r_first; r < r_last; ++r) {
        for (int k : inputs_before(g, cp.sub[r], cp.sub[r + 1])) o << "  float pf" << r << "_" << k << ";\n";
        int lo, hi;
        sub_words(g, cp.sub[r], cp.sub[r + 1], width, &lo, &hi);
        for (int q = lo; q < hi && width > 1; ++q)
            o << "  " << (width == 16 ? "emo_u32x4" : "unsigned int") << " P" << r << "L" << q << ";\n";
    }
    auto prefetch = [&](int r) {
        for (int k : inputs_before(g, cp.sub[r], cp.sub[r + 1]))
            o << "  pf" << r << "_" << k << " = EMO_AT(ck, " << cp.ck_row[k] << ");\n";
        int lo, hi;
        sub_words(g, cp.sub[r], cp.sub[r + 1], width, &lo, &hi);
        for (int q = lo; q < hi && width > 1; ++q) o << "  P" << r << "L" << q << " = rowp[" << q << "];\n";
    };
    std::vector<std::string> level_expr(g.ops.size());
    for (int r = r_last; r >= r_first; --r) {
        const int c = cp.sub[r], d = cp.sub[r + 1];
        const bool fetched = r < r_last;
        o << "  {\n";
        for (int k : inputs_before(g, c, d)) {
            if (fetched) o << "  const float f" << k << " = pf" << r << "_" << k << ";\n";
            else o << "  const float f" << k << " = EMO_AT(ck, " << cp.ck_row[k] << ");\n";
        }
        RangeOpts ro;
        ro.a = c;
        ro.b = d;
        ro.accumulate = false;
        ro.base_pack = w.base_pack;
        ro.tab_end = w.tab_end;
        ro.declare_row = false;
        ro.preload = false;
        ro.checks = false;
        ro.time_only = true;
        if (fetched && width > 1) {
            ro.pfx = "P" + std::to_string(r) + "L";
            sub_words(g, c, d, width, &ro.pre_lo, &ro.pre_hi);
        }
        LevelPlan lp = emit_forward_range(o, g, ro, &level_expr);
        lp.launder();
        bool prefetched = r == r_first;
        if (!cp.staged && !prefetched) {
            prefetch(r - 1);
            prefetched = true;
        }
        for (int i = d - 1; i >= c; --i) {
            const JitOp &op = g.ops[i];
            // table reads index through zb, and level bytes are extracted from words, that pass
            // through an empty asm every 16 steps: neither can be hoisted (each would hold a VGPR
            // from there on)
            if ((d - 1 - i) % 16 == 0) {
                std::vector<std::string> ops = {"zb"};
                if (lp.width > 1)
                    for (int k = i; k > i - 16 && k >= c; --k)
                        if (g.ops[k].pack >= 0) {
                            const std::string wd = lp.pfx + std::to_string(g.ops[k].pack / lp.width);
                            if (std::find(ops.begin(), ops.end(), wd) == ops.end()) ops.push_back(wd);
                        }
                o << "  __asm__ __volatile__(\"\" :";
                for (size_t k = 0; k < ops.size(); ++k) o << (k ? ", " : " ") << "\"+v\"(" << ops[k] << ")";
                o << ");\n";
            }
            std::string lft;
            if (op.out.empty()) {
                lft = "Tb";
            } else {
                bool have = false;
                for (int k : op.out) {
                    std::string v = "s" + std::to_string(k);
                    lft = have ? "fminf(" + lft + ", " + v + ")" : v;
                    have = true;
                }
            }
            o << "  const float lf" << i << " = " << lft << ";\n";
            std::string dur = flit(op.dur);
            if (op.pack >= 0) {
                const std::string lv = lp.width == 1 ? lp.reload_byte(op.pack) : level_expr[i];
                o << "  const float t" << i << " = tab[zb + " << lp.row_entry(op.pack) << " + "
                  << lv << "];\n";
                dur = "t" + std::to_string(i);
            }
            if (!op.in.empty()) {
                o << "  s" << i << " = lf" << i << " - " << dur << ";\n";
                if (cp.bk_row[i] >= 0) o << "  EMO_AT(bk, " << cp.bk_row[i] << ") = s" << i << ";\n";
            }
            if (op.pack >= 0) {
                const int p = op.pack;
                const std::string v = "isbad ? EMO_NAN : lf" + std::to_string(i) + " - f" + std::to_string(i);
                if (cp.staged) {
                    const int k = p % 32;
                    o << "  stg[" << k * 64 << " + (lane ^ " << 8 * (k / 4) << ")] = " << v << ";\n";
                    if (k == 0 && !prefetched) {
                        prefetch(r - 1);
                        prefetched = true;
                    }
                    if (k == 0) o << "  emo_cflush(stg, S, wbase, B, " << p << ");\n";
                } else {
                    o << "  srow[" << p << "] = " << v << ";\n";
                }
            }
        }
        if (!prefetched) prefetch(r - 1);
        o << "  }\n";
    }
    o << "}\n\n";
}

}  // namespace

std::string jit_generate_chain(const JitGraph &g, const ChainPlan &cp) {
    std::ostringstream o;
    o << "#define EMO_BLOCK " << cp.block << "\n" << kPrelude << kEmoSelectSource << "\n";
    if (cp.staged) o << chain_flush_source(g.P);
    for (int j = 0; j < cp.segments(); ++j) emit_chain_forward(o, g, cp, j);
    if (cp.slack)
        for (int j = 0; j < cp.segments(); ++j) emit_chain_backward(o, g, cp, j);
    return o.str();
}

size_t chain_scratch_bytes(const ChainPlan &cp, int64_t B) {
    const size_t bp = static_cast<size_t>(chain_pitch(B));
    return bp * (4 * static_cast<size_t>(cp.n_ck + cp.n_bk + 2) + 8);
}

// ------------------------------------------------------------------ cut-segment kernels

namespace {
constexpr size_t kCutTableLds = 32 * 1024;   // (t, e) table window of one segment in LDS

int packs_in(const JitGraph &g, int a, int b) {
    int n = 0;
    for (int i = a; i < b; ++i) n += g.ops[i].pack >= 0 ? 1 : 0;
    return n;
}
}  // namespace

CutPlan jit_cut_plan(const JitGraph &g, const std::vector<int32_t> &cuts, int max_packs, int sub_packs) {
    CutPlan cp;
    const int n = static_cast<int>(g.ops.size());
    if (cuts.empty() || !g.pack_monotone || g.P % 32 != 0) return cp;
    // a segment's (t, e) table rows stay within the LDS window (whole slack tiles of 32 packs)
    const long long fit = (static_cast<long long>(kCutTableLds / (sizeof(float) * 2)) -
                           (is_pow2(g.F) ? 0 : kTablePad)) / g.F / 32 * 32;
    max_packs = static_cast<int>(std::min<long long>(max_packs, fit));
    if (max_packs < 32) return cp;
    std::vector<int> npk_before(n + 1, 0);
    for (int i = 0; i < n; ++i) npk_before[i + 1] = npk_before[i] + (g.ops[i].pack >= 0 ? 1 : 0);
    // pieces between consecutive cuts (each ends with its cut), then the steps after the last;
    // only cuts after a multiple of 32 packs can end a segment (whole slack tiles)
    std::vector<int> ends;
    for (int c : cuts)
        if (npk_before[c + 1] % 32 == 0) ends.push_back(c + 1);
    cp.closed_last = !ends.empty() && ends.back() == n;
    if (!cp.closed_last) ends.push_back(n);
    // segments: as many whole pieces as max_packs allows
    std::vector<int32_t> seg = {0};
    int last_end = -1;
    for (int e : ends) {
        if (npk_before[e] - npk_before[seg.back()] <= max_packs) {
            last_end = e;
            continue;
        }
        if (last_end <= seg.back()) return CutPlan();   // one piece alone is too large
        seg.push_back(last_end);
        if (npk_before[e] - npk_before[last_end] > max_packs) return CutPlan();
        last_end = e;
    }
    seg.push_back(last_end);
    const int m = static_cast<int>(seg.size()) - 1;
    if (m < 2) return CutPlan();
    for (int j = 0; j < m; ++j) {
        const int a = seg[j], b = seg[j + 1];
        const bool closed = j + 1 < m || cp.closed_last;
        // no edge leaves a segment except from its final cut, and every edge into it comes from
        // the cut before it (the property the cuts were found by; checked again here)
        for (int i = a; i < b; ++i) {
            for (int k : g.ops[i].out)
                if (k >= b && !(closed && i == b - 1)) return CutPlan();
            for (int k : g.ops[i].in)
                if (k < a && k != a - 1) return CutPlan();
            if (j > 0 && g.ops[i].cst != 0.f) return CutPlan();
        }
        // slack tiles of 32 packs never straddle two segments; the table window fits in LDS
        int lo = g.P, hi = -1;
        for (int i = a; i < b; ++i)
            if (g.ops[i].pack >= 0) {
                lo = std::min(lo, g.ops[i].pack);
                hi = std::max(hi, g.ops[i].pack);
            }
        if (hi < 0 || lo % 32 != 0 || (hi + 1) % 32 != 0) return CutPlan();
        const size_t ent = static_cast<size_t>(hi - lo + 1) * g.F + (is_pow2(g.F) ? 0 : kTablePad);
        if (ent * sizeof(float) * 2 > kCutTableLds) return CutPlan();
    }
    cp.seg = seg;
    // energy blocks of 64 packs counted from each segment's start
    int rows = 0;
    for (int j = 0; j < m; ++j) {
        cp.blk0.push_back(rows);
        rows += (packs_in(g, seg[j], seg[j + 1]) + 63) / 64;
    }
    cp.blk0.push_back(rows);
    // recompute sub-segments of sub_packs packs (a multiple of 32: whole slack tiles)
    std::vector<int> sub_of(n);
    for (int j = 0; j < m; ++j) {
        const int a = seg[j], b = seg[j + 1];
        cp.sub.push_back(a);
        for (int c = a + 1, start = a; c < b; ++c)
            if (npk_before[c] - npk_before[start] >= sub_packs && (npk_before[c] - npk_before[a]) % 32 == 0) {
                cp.sub.push_back(c);
                start = c;
            }
    }
    cp.sub.push_back(n);
    for (size_t r = 0; r + 1 < cp.sub.size(); ++r)
        for (int i = cp.sub[r]; i < cp.sub[r + 1]; ++i) sub_of[i] = static_cast<int>(r);
    cp.ck.assign(n, 0);
    for (int j = 0; j < m; ++j)
        for (int i = seg[j]; i < seg[j + 1]; ++i)
            for (int k : g.ops[i].out)
                if (k < seg[j + 1] && sub_of[k] != sub_of[i]) cp.ck[i] = 1;
    return cp;
}

size_t cut_scratch_bytes(const CutPlan &cp, int64_t B) {
    const size_t bp = static_cast<size_t>(chain_pitch(B));
    return bp * 4 * static_cast<size_t>(cp.segments() + cp.blk0.back());
}

namespace {

TabWindow cut_window(const JitGraph &g, const CutPlan &cp, int j) {
    return chain_window(g, cp.seg[j], cp.seg[j + 1], kCutTableLds, sizeof(float) * 2);
}

// Whether step i's latest start time is read: some predecessor lies in its own segment.
bool reads_start(const JitGraph &g, int i, int a) {
    for (int k : g.ops[i].in)
        if (k >= a) return true;
    return false;
}

// Backward pass of segment j (slack): the sub-segments from last to first, each recomputing its
// finish times from the checkpoint copies c<k> (or 0 for the cut before the segment) and level
// words loaded again, then walking its steps backwards.  Latest finish times are local: the
// segment's makespan Db for its final cut and for sinks.
void emit_cut_backward(std::ostringstream &o, const JitGraph &g, const CutPlan &cp, int j,
                       const TabWindow &w) {
    const int a = cp.seg[j], b = cp.seg[j + 1];
    const bool closed = j + 1 < cp.segments() || cp.closed_last;
    o << "  {\n";
    o << "  const bool isbad = D != D;\n  const float Db = isbad ? 0.f : D;\n";
    o << "  unsigned int zb = 0u;\n  __asm__ __volatile__(\"\" : \"+v\"(zb));\n";
    o << "  unsigned int bad = 0u;\n  (void)bad;\n";
    o << LevelPlan::row_decl(jit_level_width(g));
    for (int i = a; i < b; ++i)
        if (reads_start(g, i, a)) o << "  float s" << i << ";\n";
    int r_first = 0;
    while (cp.sub[r_first] < a) ++r_first;
    int r_last = r_first;
    while (cp.sub[r_last + 1] < b) ++r_last;
    std::vector<std::string> level_expr(g.ops.size());
    for (int r = r_last; r >= r_first; --r) {
        const int c = cp.sub[r], d = cp.sub[r + 1];
        o << "  {\n";
        for (int k : inputs_before(g, c, d)) {
            if (k < a) o << "  const float f" << k << " = 0.f;\n";
            else o << "  const float f" << k << " = c" << k << ";\n";
        }
        RangeOpts ro;
        ro.a = c;
        ro.b = d;
        ro.accumulate = false;
        ro.base_pack = w.base_pack;
        ro.tab_end = w.tab_end;
        ro.declare_row = false;
        ro.preload = false;
        ro.checks = false;
        ro.time_only = true;
        ro.tsel = ".x";
        LevelPlan lp = emit_forward_range(o, g, ro, &level_expr);
        lp.launder();
        for (int i = d - 1; i >= c; --i) {
            const JitOp &op = g.ops[i];
            if ((d - 1 - i) % 16 == 0) {
                std::vector<std::string> ops = {"zb"};
                for (int k = i; k > i - 16 && k >= c; --k)
                    if (g.ops[k].pack >= 0) {
                        const std::string wd = lp.pfx + std::to_string(g.ops[k].pack / lp.width);
                        if (std::find(ops.begin(), ops.end(), wd) == ops.end()) ops.push_back(wd);
                    }
                o << "  __asm__ __volatile__(\"\" :";
                for (size_t k = 0; k < ops.size(); ++k) o << (k ? ", " : " ") << "\"+v\"(" << ops[k] << ")";
                o << ");\n";
            }
            std::string lft;
            if (op.out.empty() || (closed && i == b - 1)) {
                lft = "Db";
            } else {
                bool have = false;
                for (int k : op.out) {
                    std::string v = "s" + std::to_string(k);
                    lft = have ? "fminf(" + lft + ", " + v + ")" : v;
                    have = true;
                }
            }
            o << "  const float lf" << i << " = " << lft << ";\n";
            std::string dur = flit(op.dur);
            if (op.pack >= 0) {
                o << "  const float t" << i << " = tab[zb + " << lp.row_entry(op.pack) << " + "
                  << level_expr[i] << "].x;\n";
                dur = "t" + std::to_string(i);
            }
            if (reads_start(g, i, a)) o << "  s" << i << " = lf" << i << " - " << dur << ";\n";
            if (op.pack >= 0) {
                const int k = op.pack % 32;
                o << "  stg[" << k * 64 << " + (lane ^ " << 8 * (k / 4) << ")] = isbad ? EMO_NAN : lf" << i
                  << " - f" << i << ";\n";
                if (k == 0) o << "  emo_cflush(stg, S, wbase, B, " << op.pack << ");\n";
            }
        }
        o << "  }\n";
    }
    o << "  }\n";
}

// Segment j of the segment kernel: its table window, the forward pass from the local origin
// (its local makespan D and energy blocks stored), and with slack the backward pass.
void emit_cut_segment(std::ostringstream &o, const JitGraph &g, const CutPlan &cp, int j, bool slack) {
    const int a = cp.seg[j], b = cp.seg[j + 1];
    const bool closed = j + 1 < cp.segments() || cp.closed_last;
    const TabWindow w = cut_window(g, cp, j);
    int plo = g.P, phi = -1;
    for (int i = a; i < b; ++i)
        if (g.ops[i].pack >= 0) {
            plo = std::min(plo, g.ops[i].pack);
            phi = std::max(phi, g.ops[i].pack);
        }
    const int width = jit_level_width(g);
    const int q_lo = plo / width, q_hi = phi / width + 1;
    o << "  case " << j << ": {\n";
    if (slack) {
        o << table_copy(w.entries, w.base_pack * g.F, 8, cp.block) << "  __syncthreads();\n";
        o << "  {\n";
        o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
    } else {
        // forward only: the segment's level words are requested before the table window is
        // copied, so that the copy and its barrier overlap their latency (in the slack kernel
        // this order was slower: 1.44 vs 1.29 ms on the 4096-pack workload)
        o << "  {\n";
        o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
        o << LevelPlan::row_decl(width);
        for (int q = q_lo; q < q_hi; ++q)
            o << "  " << (width == 16 ? "emo_u32x4" : "unsigned int") << " L" << q << " = rowp[" << q << "];\n";
        o << table_copy(w.entries, w.base_pack * g.F, 8, cp.block) << "  __syncthreads();\n";
    }
    if (slack)
        for (int i = a; i < b; ++i)
            if (cp.ck[i]) o << "  float c" << i << ";\n";
    o << "  float D;\n  {\n";
    o << "  unsigned int bad = 0u;\n  float eb = 0.f;\n  float T = 0.f;\n";
    if (j > 0) o << "  const float f" << a - 1 << " = 0.f;\n";
    RangeOpts r;
    r.a = a;
    r.b = b;
    r.npk0 = 0;
    r.blk_row0 = cp.blk0[j];
    r.base_pack = w.base_pack;
    r.tab_end = w.tab_end;
    r.declare_row = slack;
    r.preload = false;
    r.pre_lo = slack ? 0 : q_lo;
    r.pre_hi = slack ? 0 : q_hi;
    r.ck_copy = slack ? &cp.ck : nullptr;
    LevelPlan lp = emit_forward_range(o, g, r, nullptr);
    const int npk = packs_in(g, a, b);
    if (npk % 64) o << "  EMO_AT(Ebg, " << cp.blk0[j] + npk / 64 << ") = eb;\n";
    o << "  D = " << (closed ? "f" + std::to_string(b - 1) : std::string("T")) << ";\n";
    o << "  if ((bad & " << lp.bad_bits() << ") != 0u) D = EMO_NAN;\n";
    o << "  EMO_AT(Dg, " << j << ") = D;\n  }\n";
    if (slack) emit_cut_backward(o, g, cp, j, w);
    o << "  }\n  } break;\n";
}

}  // namespace

std::string jit_generate_cut(const JitGraph &g, const CutPlan &cp) {
    std::ostringstream o;
    o << "#define EMO_BLOCK " << cp.block << "\n" << kPrelude << kEmoSelectSource << "\n";
    o << chain_flush_source(g.P);
    long long entries = 0;   // the largest window, so that every segment kernel has one LDS layout
    for (int j = 0; j < cp.segments(); ++j) entries = std::max(entries, cut_window(g, cp, j).entries);
    for (int slack = 0; slack < 2; ++slack)
      for (int kk = 0; kk < (slack ? cp.kernels() : cp.kernels_fwd()); ++kk) {
        const int per = slack ? cp.per_kernel : cp.per_kernel_fwd;
        const int j0 = kk * per, j1 = std::min(cp.segments(), j0 + per);
        o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
          << (slack ? "emo_ks" : "emo_kf") << kk
          << "(const u8 *__restrict__ lv, long long B, long long bp,\n"
             "    const float2 *__restrict__ tabg, float *__restrict__ Dg, float *__restrict__ Ebg,\n"
             "    float *__restrict__ S) {\n";
        // the table first, at LDS address 0: every table read keeps its row offset as an
        // immediate (16 bits), which a table placed after the 64 KB of slack tiles would not
        if (slack)
            o << "  __shared__ struct { float2 t[" << entries << "]; float s[EMO_BLOCK / 64][32 * 64]; } emo_sh;\n"
                 "  float2 *tab = emo_sh.t;\n"
                 "  float *stg = emo_sh.s[threadIdx.x / EMO_WAVE];\n";
        else
            o << "  __shared__ float2 tab[" << entries << "];\n";
        o << chain_lanes(cp.block);
        o << "  const int lane = threadIdx.x % EMO_WAVE;\n"
             "  const long long wbase = (long long)blockIdx.x * EMO_BLOCK + (threadIdx.x / EMO_WAVE) * EMO_WAVE;\n"
             "  (void)lane; (void)wbase; (void)S;\n";
        o << "  switch (blockIdx.y + " << j0 << ") {\n";
        for (int j = j0; j < j1; ++j) emit_cut_segment(o, g, cp, j, slack != 0);
        o << "  default: break;\n  }\n}\n\n";
      }
    // finishing kernel: makespan = the segments' local makespans added in order, energy = the
    // blocks added in order into fp64 plus static power times makespan (Eq. 2); an invalid level
    // in any segment (NaN D) makes the candidate's makespan, energy and slack row NaN
    o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
         "emo_kfin(long long B, long long bp, const float *__restrict__ Dg, const float *__restrict__ Ebg,\n"
         "    float *__restrict__ S, float *__restrict__ To, float *__restrict__ Eo, EmoTargets tg) {\n";
    o << chain_lanes(cp.block);
    o << "  float T = EMO_AT(Dg, 0);\n";
    for (int j = 1; j < cp.segments(); ++j) o << "  T = T + EMO_AT(Dg, " << j << ");\n";
    o << "  const bool isbad = T != T;\n";
    o << "  T = fmaxf(T, " << flit(g.t_const) << ");\n";
    o << "  double ed = 0.0;\n";
    for (int q = 0; q < cp.blk0.back(); ++q) o << "  ed += (double)EMO_AT(Ebg, " << q << ");\n";
    o << "  float E = (float)(ed + (double)" << flit(g.static_power) << " * (double)T);\n";
    o << "  if (isbad) { T = EMO_NAN; E = EMO_NAN; }\n";
    o << "  if (active) { if (To) To[cand] = T; if (Eo) Eo[cand] = E; }\n";
    o << "  if (S) {\n"
         "    const int lane = threadIdx.x % EMO_WAVE;\n"
         "    const long long wbase = (long long)blockIdx.x * EMO_BLOCK + (threadIdx.x / EMO_WAVE) * EMO_WAVE;\n"
         "    unsigned long long bm = __ballot(active && isbad);\n"
         "    while (bm) {\n"
         "      const int r = __ffsll((long long)bm) - 1;\n"
         "      bm &= bm - 1ull;\n"
         "      float *__restrict__ srow = S + (wbase + r) * " << g.P << "LL;\n"
         "      for (int c = 4 * lane; c < " << g.P << "; c += 4 * EMO_WAVE) *(emo_f32x4 *)(srow + c) = (emo_f32x4)(EMO_NAN);\n"
         "    }\n"
         "  }\n";
    o << "  if (tg.n) emo_select_all(blockIdx.x, active, T, E, cand, B, tg);\n";
    o << "}\n";
    return o.str();
}

namespace {

// Compiles `src` for gfx950 and loads it as a module.  0 on success, 1 compile error, 2 load error.
int compile_module(const std::string &src, hipModule_t *module, double *seconds, std::string *log) {
    hiprtcProgram prog;
    if (hiprtcCreateProgram(&prog, src.c_str(), "emo_specialised.hip", 0, nullptr, nullptr) !=
        HIPRTC_SUCCESS) {
        *log = "hiprtcCreateProgram failed";
        return 1;
    }
    const char *opts[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                          "-Xclang", "-packed-fp32-ops"};
    auto t0 = std::chrono::steady_clock::now();
    hiprtcResult r = hiprtcCompileProgram(prog, sizeof(opts) / sizeof(opts[0]), opts);
    *seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    size_t ls = 0;
    hiprtcGetProgramLogSize(prog, &ls);
    if (ls > 1) {
        std::string l(ls, '\0');
        hiprtcGetProgramLog(prog, &l[0]);
        *log = l;
    }
    if (r != HIPRTC_SUCCESS) {
        hiprtcDestroyProgram(&prog);
        if (log->empty()) *log = hiprtcGetErrorString(r);
        return 1;
    }
    size_t cs = 0;
    hiprtcGetCodeSize(prog, &cs);
    std::string code(cs, '\0');
    hiprtcGetCode(prog, &code[0]);
    hiprtcDestroyProgram(&prog);
    hipError_t e = hipModuleLoadData(module, code.data());
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *log = std::string("hipModuleLoadData: ") + hipGetErrorString(e);
        *module = nullptr;
        return 2;
    }
    return 0;
}

bool get_function(hipModule_t m, const std::string &name, hipFunction_t *f) {
    if (hipModuleGetFunction(f, m, name.c_str()) == hipSuccess) return true;
    (void)hipGetLastError();   // clear the runtime's sticky error
    return false;
}

}  // namespace

int jit_compile(const std::string &src, bool with_slack, JitModule *out, std::string *log) {
    int rc = compile_module(src, &out->module, &out->compile_seconds, log);
    if (rc != 0) return rc;
    if (!get_function(out->module, "emo_sp_select", &out->select) ||
        (with_slack && !get_function(out->module, "emo_sp_slack", &out->slack))) {
        *log = "specialised kernels missing from the module";
        (void)hipModuleUnload(out->module);
        *out = JitModule();
        return 2;
    }
    return 0;
}

int jit_compile_chain(const std::string &src, const ChainPlan &cp, JitModule *out, std::string *log) {
    int rc = compile_module(src, &out->module, &out->compile_seconds, log);
    if (rc != 0) return rc;
    out->chain = true;
    out->plan = cp;
    out->block = cp.block;
    out->cf.assign(cp.segments(), nullptr);
    out->cb.assign(cp.slack ? cp.segments() : 0, nullptr);
    bool okf = true;
    for (int j = 0; j < cp.segments(); ++j) {
        okf = okf && get_function(out->module, "emo_cf" + std::to_string(j), &out->cf[j]);
        if (cp.slack) okf = okf && get_function(out->module, "emo_cb" + std::to_string(j), &out->cb[j]);
    }
    if (!okf) {
        *log = "segmented kernels missing from the module";
        (void)hipModuleUnload(out->module);
        *out = JitModule();
        return 2;
    }
    return 0;
}

int jit_compile_cut(const std::string &src, const CutPlan &cp, JitModule *out, std::string *log) {
    int rc = compile_module(src, &out->module, &out->compile_seconds, log);
    if (rc != 0) return rc;
    out->cut = true;
    out->cut_plan = cp;
    out->block = cp.block;
    out->kf.assign(cp.kernels_fwd(), nullptr);
    out->ks.assign(cp.kernels(), nullptr);
    bool okf = get_function(out->module, "emo_kfin", &out->kfin);
    for (int k = 0; k < cp.kernels_fwd(); ++k)
        okf = okf && get_function(out->module, "emo_kf" + std::to_string(k), &out->kf[k]);
    for (int k = 0; k < cp.kernels(); ++k)
        okf = okf && get_function(out->module, "emo_ks" + std::to_string(k), &out->ks[k]);
    if (!okf) {
        *log = "cut-segment kernels missing from the module";
        (void)hipModuleUnload(out->module);
        *out = JitModule();
        return 2;
    }
    return 0;
}

void jit_unload(JitModule *m) {
    if (m->module) (void)hipModuleUnload(m->module);
    *m = JitModule();
}

namespace {
unsigned grid_of(int64_t B, int block) { return static_cast<unsigned>((B + block - 1) / block); }
}  // namespace

int jit_compile_intervals(const std::string &src, JitModule *out, std::string *log) {
    int rc = compile_module(src, &out->module, &out->compile_seconds, log);
    if (rc != 0) return rc;
    int dev = 0;
    if (!get_function(out->module, "emo_iv", &out->select) ||
        hipFuncGetAttribute(&out->iv_static_lds, HIP_FUNC_ATTRIBUTE_SHARED_SIZE_BYTES, out->select) !=
            hipSuccess ||
        hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&out->iv_max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
            hipSuccess) {
        (void)hipGetLastError();
        *log = "time-interval kernel missing from the module or its attributes unknown";
        (void)hipModuleUnload(out->module);
        *out = JitModule();
        return 2;
    }
    return 0;
}

size_t jit_iv_dyn_lds(int block, int K, int M) {
    const size_t sd = static_cast<size_t>(((K + 3) >> 2) | 1);
    return static_cast<size_t>(M) * 8 + static_cast<size_t>(block) * sd * 4;
}

int64_t jit_blocks(const JitModule &m, int64_t B) { return grid_of(B, m.block); }

namespace {
int64_t resident_blocks(hipFunction_t f, int block) {
    int dev = 0, ncu = 0, nb = 0;
    if (!f || hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&nb, f, block, 0) != hipSuccess || nb < 1) {
        (void)hipGetLastError();
        return 0;   // unknown: one workgroup per group
    }
    return static_cast<int64_t>(nb) * ncu;
}

unsigned capped_grid(int64_t B, int block, int64_t cap) {
    const int64_t groups = (B + block - 1) / block;
    return static_cast<unsigned>(cap > 0 ? std::min(groups, cap) : groups);
}
}  // namespace

void jit_set_caps(JitModule *m) {
    m->select_cap = resident_blocks(m->select, m->block);
    m->slack_cap = resident_blocks(m->slack, m->block);
}

hipError_t jit_launch_intervals(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                                const IvJitArgs &a, int64_t cap, float *T, float *E, const SelTargets &tg,
                                hipStream_t s) {
    SelTargets dt = tg;
    long long b = B;
    IvJitArgs args_v = a;
    const uintptr_t al = reinterpret_cast<uintptr_t>(levels);
    int copy = a.K % 16 == 0 && al % 16 == 0 ? 16 : (a.K % 4 == 0 && al % 4 == 0 ? 4 : 1);
    float inv_k = static_cast<float>(1.0 / a.K);
    void *args[] = {&levels, &b, &tab, &args_v, &copy, &inv_k, &T, &E, &dt};
    const unsigned dyn = static_cast<unsigned>(jit_iv_dyn_lds(m.block, a.K, a.M));
    return hipModuleLaunchKernel(m.select, capped_grid(B, m.block, cap), 1, 1, m.block, 1, 1, dyn, s, args,
                                 nullptr);
}

int64_t jit_iv_cap(const JitModule &m, int K, int M) {
    int dev = 0, ncu = 0, nb = 0;
    const size_t dyn = jit_iv_dyn_lds(m.block, K, M);
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipModuleOccupancyMaxActiveBlocksPerMultiprocessor(&nb, m.select, m.block, dyn) != hipSuccess ||
        nb < 1) {
        (void)hipGetLastError();
        return 0;
    }
    return static_cast<int64_t>(nb) * ncu;
}

hipError_t jit_launch_forward(const JitModule &m, const uint8_t *levels, int64_t B,
                              const float2 *tab, float *T, float *E, const SelTargets &tg, hipStream_t s) {
    long long b = B;
    SelTargets dt = tg;
    void *args[] = {&levels, &b, &tab, &T, &E, &dt};
    return hipModuleLaunchKernel(m.select, capped_grid(B, m.block, m.select_cap), 1, 1, m.block, 1, 1, 0,
                                 s, args, nullptr);
}

int64_t jit_chain_blocks(const JitModule &m, int64_t B) { return grid_of(B, m.plan.block); }

hipError_t jit_launch_chain(const JitModule &m, const uint8_t *levels, int64_t B,
                            const float2 *tab, const float *tabt, void *scratch, float *S,
                            float *T, float *E, const SelTargets &tg, hipStream_t s) {
    const ChainPlan &cp = m.plan;
    const unsigned grid = grid_of(B, cp.block);
    const unsigned bgrid = grid_of(B, cp.bblock);
    long long bp = chain_pitch(B);
    float *ck = static_cast<float *>(scratch);
    float *bk = ck + static_cast<size_t>(cp.n_ck) * bp;
    float *Tc = bk + static_cast<size_t>(cp.n_bk) * bp;
    float *Ebc = Tc + bp;
    double *Edc = reinterpret_cast<double *>(Ebc + bp);   // 8-byte aligned: bp is a multiple of 64
    long long b = B;
    int full = S ? 1 : 0;
    const int m_seg = cp.segments();
    for (int j = 0; j < m_seg; ++j) {
        const bool last = j + 1 == m_seg;
        float *To = last ? T : nullptr;
        float *Eo = last ? E : nullptr;
        SelTargets dt = last ? tg : SelTargets();
        void *args[] = {&levels, &b, &bp, &tab, &ck, &Tc, &Edc, &Ebc, &full, &To, &Eo, &dt};
        hipError_t e = hipModuleLaunchKernel(m.cf[j], grid, 1, 1, cp.block, 1, 1, 0, s, args, nullptr);
        if (e != hipSuccess) return e;
    }
    if (!S) return hipSuccess;
    for (int j = m_seg - 1; j >= 0; --j) {
        const float *ckc = ck, *Tcc = Tc;
        void *args[] = {&levels, &b, &bp, &tabt, &ckc, &Tcc, &bk, &S};
        hipError_t e = hipModuleLaunchKernel(m.cb[j], bgrid, 1, 1, cp.bblock, 1, 1, 0, s, args, nullptr);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

int64_t jit_cut_blocks(const JitModule &m, int64_t B) { return grid_of(B, m.cut_plan.block); }

hipError_t jit_launch_cut(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                          void *scratch, float *S, float *T, float *E, const SelTargets &tg, hipStream_t s) {
    const CutPlan &cp = m.cut_plan;
    const unsigned grid = grid_of(B, cp.block);
    long long bp = chain_pitch(B);
    float *Dg = static_cast<float *>(scratch);
    float *Ebg = Dg + static_cast<size_t>(cp.segments()) * bp;
    long long b = B;
    void *args[] = {&levels, &b, &bp, &tab, &Dg, &Ebg, &S};
    const int per = S ? cp.per_kernel : cp.per_kernel_fwd;
    const int nk = S ? cp.kernels() : cp.kernels_fwd();
    for (int k = 0; k < nk; ++k) {
        const int rows = std::min(per, cp.segments() - k * per);
        hipError_t e = hipModuleLaunchKernel(S ? m.ks[k] : m.kf[k], grid, static_cast<unsigned>(rows), 1,
                                             cp.block, 1, 1, 0, s, args, nullptr);
        if (e != hipSuccess) return e;
    }
    const float *Dc = Dg, *Ec = Ebg;
    SelTargets dt = tg;
    void *fargs[] = {&b, &bp, &Dc, &Ec, &S, &T, &E, &dt};
    return hipModuleLaunchKernel(m.kfin, grid, 1, 1, cp.block, 1, 1, 0, s, fargs, nullptr);
}

hipError_t jit_launch_slack(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                            float *S, float *T, float *E, const SelTargets &tg, hipStream_t s) {
    long long b = B;
    SelTargets dt = tg;
    void *args[] = {&levels, &b, &tab, &S, &T, &E, &dt};
    return hipModuleLaunchKernel(m.slack, capped_grid(B, m.block, m.slack_cap), 1, 1, m.block, 1, 1, 0,
                                 s, args, nullptr);
}

}  // namespace emo
