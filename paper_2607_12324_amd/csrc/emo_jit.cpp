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
    std::vector<char> loaded, released;
    std::ostringstream *o;
    // Level words are loaded a whole 128-byte line of the row at a time (all of a group's
    // loads back to back, so the line is fetched from L2 once) and one group ahead of use.
    static constexpr int kGroupBytes = 128;

    int group_words() const { return kGroupBytes / width; }

    unsigned fmask() const { return static_cast<unsigned>(F - 1) * 0x01010101u; }
    int nwords() const { return (P + width - 1) / width; }

    void check(const std::string &w) {
        if (F >= 256) return;
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

    void begin() {
        if (width == 16) *o << "  const uint4 *rowp = (const uint4 *)row;\n";
        else if (width == 4) *o << "  const unsigned int *rowp = (const unsigned int *)row;\n";
        loaded.assign(nwords() + 1, 0);
        released.assign(nwords() + 1, 0);
        if (width == 1) return;
        load_group(0);
    }

    void load(int q) {
        if (q >= nwords() || loaded[q]) return;
        loaded[q] = 1;
        *o << "  " << (width == 16 ? "uint4" : "unsigned int") << " L" << q << " = rowp[" << q << "];\n";
    }

    void load_group(int gidx) {
        for (int q = gidx * group_words(); q < (gidx + 1) * group_words(); ++q) load(q);
    }

    bool needs_release(int p) const { return width != 1 && !released[p / width]; }

    // Releases chunk q.  `ride` names values computed before this point (the energy partial
    // sum and the finish times still needed later) that pass through the same barrier, so the
    // arithmetic of the previous chunk completes before this chunk's table reads start.
    void release(int q, const std::vector<std::string> &ride) {
        const int gidx = q / group_words();
        if (!loaded[q] || (q % group_words() == 0 && (gidx + 1) * group_words() < nwords() &&
                           !loaded[(gidx + 1) * group_words()])) {
            *o << "  __asm__ __volatile__(\"\" : \"+v\"(rowp));\n";
            load_group(gidx);
            load_group(gidx + 1);
        }
        std::string w = "L" + std::to_string(q);
        std::vector<std::string> ops;
        if (width == 16) {
            for (int k = 0; k < 4; ++k) ops.push_back(w + "." + comp(k));
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

    // Returns the expression of pack p's level byte (emitting loads and checks as needed).
    std::string byte_of(int p) {
        std::ostringstream e;
        if (width == 1) {
            *o << "  const unsigned int B" << p << " = row[" << p << "];\n";
            if (F < 256) *o << "  bad |= (B" << p << " >= " << F << "u) ? 0x80808080u : 0u;\n";
            if (pow2 && F < 256 && !raw_ok(p)) e << "(B" << p << " & " << (F - 1) << "u)";
            else e << "B" << p;
            return e.str();
        }
        const int q = p / width;
        std::string w = "L" + std::to_string(q);
        if (width == 16) w += std::string(".") + comp((p % 16) / 4);
        const unsigned m = (pow2 && F < 256 && !raw_ok(p)) ? static_cast<unsigned>(F - 1) : 0xffu;
        e << "((" << w << " >> " << 8 * (p % 4) << ") & " << m << "u)";
        return e.str();
    }

    // Whether any byte value at pack p indexes inside the unpadded table.
    bool raw_ok(int p) const { return !pow2 || static_cast<long long>(p) * F + 255 < static_cast<long long>(P) * F; }

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

// Forward pass: declares f<i> (finish time) for every step, and T, E, bad; records the
// expression of each pack step's level byte in *level_expr.
void emit_forward(std::ostringstream &o, const JitGraph &g, std::vector<std::string> *level_expr) {
    LevelPlan lp;
    lp.P = g.P;
    lp.F = g.F;
    lp.width = jit_level_width(g.P);
    lp.pow2 = is_pow2(g.F);
    lp.o = &o;
    o << "  unsigned int bad = 0u;\n  float eb = 0.f;\n  double ed = 0.0;\n";
    lp.begin();
    o << "  float T = " << flit(g.t_const) << ";\n";
    int npk = 0;
    const int n = static_cast<int>(g.ops.size());
    std::vector<int> last_use(n, -1);
    for (int i = 0; i < n; ++i)
        for (int k : g.ops[i].in) last_use[k] = std::max(last_use[k], i);
    int since = 0;   // first step not yet passed through a barrier
    for (int i = 0; i < n; ++i) {
        const JitOp &op = g.ops[i];
        if (op.pack >= 0 && lp.needs_release(op.pack)) {
            std::vector<std::string> ride = {"eb", "ed", "bad"};
            for (int j = since; j < i; ++j)
                if (last_use[j] >= i) ride.push_back("f" + std::to_string(j));
            lp.release(op.pack / lp.width, ride);
            since = i;
        }
        if (op.pack >= 0) {
            std::string b = lp.byte_of(op.pack);
            if (level_expr) (*level_expr)[i] = b;
            o << "  const float2 te" << i << " = tab[" << static_cast<long long>(op.pack) * g.F
              << " + " << b << "];\n";
            o << "  float f" << i << " = " << est_expr(g, i, "f") << " + te" << i << ".x;\n";
            o << "  eb += te" << i << ".y;\n";
            if (++npk % 64 == 0) o << "  ed += (double)eb;\n  eb = 0.f;\n";
        } else {
            o << "  float f" << i << " = " << est_expr(g, i, "f") << " + " << flit(op.dur) << ";\n";
        }
        if (op.out.empty()) o << "  T = fmaxf(T, f" << i << ");\n";
    }
    o << "  ed += (double)eb;\n";
    o << "  float E = (float)(ed + (double)" << flit(g.static_power) << " * (double)T);\n";
    o << "  const bool isbad = (bad & " << lp.bad_bits() << ") != 0u;\n";
    o << "  if (isbad) { T = __builtin_nanf(\"\"); E = __builtin_nanf(\"\"); }\n";
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

const char *kPrelude = R"(
typedef unsigned char u8;
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
    o << "#define EMO_LANE_SETUP \\\n"
         "  const long long gid = (long long)blockIdx.x * EMO_BLOCK + threadIdx.x; \\\n"
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
         "              float target, unsigned int *__restrict__ mask, EmoPartial *part) {\n"
         "  EMO_TABLE_DECL\n  EMO_LANE_SETUP\n"
         "  const EmoFwd r = emo_forward(lv + cand * "
      << g.P << "LL, tab);\n"
         "  if (active) { if (To) To[cand] = r.T; if (Eo) Eo[cand] = r.E; }\n"
         "  if (mask || part) emo_select_block(active, r.T, r.E, cand, B, target, mask, part);\n"
         "}\n";

    if (with_slack) {
        const bool staged = g.pack_monotone && g.P % 16 == 0;
        if (staged) {
            const int kc = stage_chunk(g.P);
            o << "#define EMO_KC " << kc << "\n";
            o << R"(
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
    if (row < B) *(float4 *)(S + row * )" << g.P << R"(LL + p0 + 4 * part) = v;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}
)";
        }
        o << "extern \"C\" __global__ void __launch_bounds__(EMO_BLOCK)\n"
             "emo_sp_slack(const u8 *__restrict__ lv, long long B, const float2 *__restrict__ tabg,\n"
             "             float *__restrict__ S, float *__restrict__ To, float *__restrict__ Eo,\n"
             "             float target, unsigned int *__restrict__ mask, EmoPartial *part) {\n"
             "  EMO_TABLE_DECL\n  EMO_LANE_SETUP\n"
             "  const int lane = threadIdx.x % EMO_WAVE;\n"
             "  const int wave = threadIdx.x / EMO_WAVE;\n"
             "  const long long wbase = (long long)blockIdx.x * EMO_BLOCK + wave * EMO_WAVE;\n"
             "  (void)lane; (void)wbase;\n";
        if (staged) {
            o << "  __shared__ float stg_all[EMO_WAVES_PER_BLOCK][EMO_KC * 65];\n"
                 "  __shared__ unsigned int bad_all[EMO_WAVES_PER_BLOCK][EMO_WAVE];\n"
                 "  float *stg = stg_all[wave];\n"
                 "  unsigned int *stg_bad = bad_all[wave];\n";
        }
        o << "  const u8 *__restrict__ row = lv + cand * " << g.P << "LL;\n";
        std::vector<std::string> level_expr(g.ops.size());
        emit_forward(o, g, &level_expr);
        o << "  if (active) { if (To) To[cand] = T; if (Eo) Eo[cand] = E; }\n";
        if (staged) o << "  stg_bad[lane] = isbad ? 1u : 0u;\n";
        emit_backward(o, g, staged, level_expr);
        o << "  if (mask || part) emo_select_block(active, T, E, cand, B, target, mask, part);\n";
        o << "}\n";
    }
    return o.str();
}

int jit_compile(const std::string &src, bool with_slack, JitModule *out, std::string *log) {
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
    out->compile_seconds =
        std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
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
    hipError_t e = hipModuleLoadData(&out->module, code.data());
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *log = std::string("hipModuleLoadData: ") + hipGetErrorString(e);
        out->module = nullptr;
        return 2;
    }
    if (hipModuleGetFunction(&out->select, out->module, "emo_sp_select") != hipSuccess ||
        (with_slack && hipModuleGetFunction(&out->slack, out->module, "emo_sp_slack") != hipSuccess)) {
        (void)hipGetLastError();   // clear the runtime's sticky error
        *log = "specialised kernels missing from the module";
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

int64_t jit_blocks(const JitModule &m, int64_t B) { return grid_of(B, m.block); }

hipError_t jit_launch_forward(const JitModule &m, const uint8_t *levels, int64_t B,
                              const float2 *tab, float *T, float *E, float target, uint32_t *mask,
                              void *part, hipStream_t s) {
    long long b = B;
    void *args[] = {&levels, &b, &tab, &T, &E, &target, &mask, &part};
    return hipModuleLaunchKernel(m.select, grid_of(B, m.block), 1, 1, m.block, 1, 1, 0, s, args, nullptr);
}

hipError_t jit_launch_slack(const JitModule &m, const uint8_t *levels, int64_t B, const float2 *tab,
                            float *S, float *T, float *E, float target, uint32_t *mask,
                            void *part, hipStream_t s) {
    long long b = B;
    void *args[] = {&levels, &b, &tab, &S, &T, &E, &target, &mask, &part};
    return hipModuleLaunchKernel(m.slack, grid_of(B, m.block), 1, 1, m.block, 1, 1, 0, s, args, nullptr);
}

}  // namespace emo
