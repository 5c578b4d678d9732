/*
 * NDVM CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, per-lane scalar interpreter of the NDVB stack bytecode with
 * a define-by-run Wengert list and an explicit reverse sweep.  It exists to
 * check the GPU path and is linked or executed only by the tests, by the
 * package smoke check and by the benchmark's CPU-baseline leg.  It shares no
 * code, header or table with the GPU path: it parses the bytecode itself and
 * never builds a lane-invariant tape.
 *
 * What it computes (paper Section 2 problem statement, Section 4 Property 1):
 * for every lane l with parameter vector theta_l it runs the program with real
 * fp64 values, taking each numeric branch the way that lane's values decide
 * (only the taken arm executes), appends one node per numeric primitive
 * (Section 3.4: structural words record nothing), and then sweeps the node
 * list in reverse applying the vector-Jacobian products of Appendix C, table
 * tab:adjoints, to obtain d loss / d theta_l along the realized trace.
 *
 * Readings where the paper leaves freedom:
 *  - sqrt/log clamp at 1e-8 in the forward, adjoint only when the argument
 *    is strictly above the clamp (table tab:adjoints caption);
 *  - single-argument sub/div are negation/reciprocal; binary div adjoint of
 *    the denominator uses the paper's form g*z/b;
 *  - sign(0) = 0 for abs;
 *  - a node whose incoming adjoint is exactly zero in every element
 *    contributes nothing (the gating that keeps untaken arms and dead lanes
 *    from polluting gradients, Section 6 lane-masking paragraph);
 *  - contractions (dot, matmul, outer, scale-adjoint) are fused
 *    multiply-add chains over the summation index in ascending order, the
 *    first term a plain product; every other operation is one IEEE
 *    operation, built with -ffp-contract=off;
 *  - 2x2 inverse is adj(A) times r = 1/det, det = a*d - b*c; det/logdet
 *    adjoints use that inverse (the "A^-1 cached in forward" of the table);
 *  - a < b is strict; unordered compares take the ELSE arm; the compare
 *    operands receive no adjoint (Property 1).
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared -pthread (-lm).
 * Compiled a second time with -DORACLE_LONG_DOUBLE the same source evaluates
 * in x87 extended precision (entry points suffixed _ld); that copy is used
 * only to estimate how much a lane's fp64 result is disturbed by rounding.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#ifdef ORACLE_LONG_DOUBLE
typedef long double real;
#define R_EXP expl
#define R_LOG logl
#define R_SQRT sqrtl
#define R_SIN sinl
#define R_COS cosl
#define R_POW powl
#define R_FABS fabsl
#define R_FMA fmal
#define ENTRY(name) name##_ld
#else
typedef double real;
#define R_EXP exp
#define R_LOG log
#define R_SQRT sqrt
#define R_SIN sin
#define R_COS cos
#define R_POW pow
#define R_FABS fabs
#define R_FMA fma
#define ENTRY(name) name
#endif

/* bytecode opcodes (NDVB format) */
enum {
    B_HALT = 0x00, B_PUSH = 0x01, B_PARAM = 0x02, B_OBS = 0x03, B_OBSX = 0x04,
    B_LOADL = 0x05, B_STOREL = 0x06, B_DUP = 0x07, B_SWAP = 0x08, B_DROP = 0x09,
    B_OVER = 0x0A,
    B_ADD = 0x10, B_SUB = 0x11, B_MUL = 0x12, B_DIV = 0x13, B_NEG = 0x14,
    B_EXP = 0x18, B_LOG = 0x19, B_SQRT = 0x1A, B_SIN = 0x1B, B_COS = 0x1C,
    B_POW = 0x1D, B_ABS = 0x1E,
    B_DOT = 0x20, B_MATMUL = 0x21, B_TRANSPOSE = 0x22, B_INV = 0x23,
    B_DET = 0x24, B_LOGDET = 0x25, B_TRACE = 0x26, B_OUTER = 0x27,
    B_PACK = 0x28, B_INDEX = 0x29,
    B_LOOP = 0x30, B_ENDLOOP = 0x31, B_IFLT = 0x32, B_ELSE = 0x33, B_ENDIF = 0x34
};

/* node kinds beyond the bytecode opcodes */
enum { K_PARAM = 0x100, K_LEAF = 0x101 };

enum { OK = 0, E_ARG = 1, E_BYTECODE = 2, E_RUNTIME = 3, E_NOMEM = 5 };

#define CLAMP_EPS ((real)1e-8)
#define MAXE 16

typedef struct { int rows, cols; real e[MAXE]; } Val;

typedef struct {
    int kind;       /* bytecode opcode of the primitive, K_PARAM or K_LEAF */
    int in[2];      /* input nodes (-1 if unused) */
    int npack;      /* PACK: number of inputs, stored in pack_in */
    int *pack_in;
    int aux;        /* INDEX: flattened element index */
    Val v;
} Node;

typedef struct {
    const uint8_t *code;     /* n_instr 8-byte words */
    const double *consts;
    uint32_t n_params, n_obs, n_instr, n_consts;
    int32_t *match;          /* LOOP<->ENDLOOP, IFLT->ELSE, ELSE->ENDIF */
    int n_locals;
} Prog;

static __thread char g_err[256];
static char g_err_shared[256];
static pthread_mutex_t g_err_mu = PTHREAD_MUTEX_INITIALIZER;

static void set_err(const char *msg, int pc) {
    snprintf(g_err, sizeof g_err, "%s (pc=%d)", msg, pc);
    pthread_mutex_lock(&g_err_mu);
    memcpy(g_err_shared, g_err, sizeof g_err_shared);
    pthread_mutex_unlock(&g_err_mu);
}

const char *ENTRY(ndvm_oracle_error)(void) { return g_err_shared; }

static uint32_t rd32(const uint8_t *p) {
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}
static int w_op(const Prog *P, int pc) { return P->code[8 * pc]; }
static int w_a(const Prog *P, int pc) { return P->code[8 * pc + 1]; }
static int w_b(const Prog *P, int pc) { return P->code[8 * pc + 2] | (P->code[8 * pc + 3] << 8); }
static uint32_t w_imm(const Prog *P, int pc) { return rd32(P->code + 8 * pc + 4); }

/* Parse the header and pair up the block words; -1 on malformed input. */
static int parse(const uint8_t *bc, size_t n, Prog *P) {
    memset(P, 0, sizeof *P);
    if (n < 24 || memcmp(bc, "NDVB", 4) != 0 || rd32(bc + 4) != 1) {
        set_err("bad NDVB header", -1);
        return -1;
    }
    P->n_params = rd32(bc + 8);
    P->n_obs = rd32(bc + 12);
    P->n_instr = rd32(bc + 16);
    P->n_consts = rd32(bc + 20);
    if ((uint64_t)24 + 8ull * P->n_instr + 8ull * P->n_consts != n) {
        set_err("NDVB size mismatch", -1);
        return -1;
    }
    P->code = bc + 24;
    P->consts = (const double *)(bc + 24 + 8ull * P->n_instr);
    P->match = (int32_t *)malloc(sizeof(int32_t) * (P->n_instr + 1));
    int32_t *stk = (int32_t *)malloc(sizeof(int32_t) * (P->n_instr + 1));
    int sp = 0, maxloc = -1;
    for (uint32_t pc = 0; pc < P->n_instr; ++pc) {
        int op = w_op(P, pc);
        P->match[pc] = -1;
        if (op == B_LOOP || op == B_IFLT) {
            stk[sp++] = (int32_t)pc;
        } else if (op == B_ELSE) {
            if (sp == 0 || w_op(P, stk[sp - 1]) != B_IFLT) { set_err("ELSE without IFLT", pc); goto bad; }
            P->match[stk[sp - 1]] = (int32_t)pc;
            stk[sp - 1] = (int32_t)pc;
        } else if (op == B_ENDIF) {
            if (sp == 0 || w_op(P, stk[sp - 1]) != B_ELSE) { set_err("ENDIF without ELSE", pc); goto bad; }
            P->match[stk[sp - 1]] = (int32_t)pc;
            sp--;
        } else if (op == B_ENDLOOP) {
            if (sp == 0 || w_op(P, stk[sp - 1]) != B_LOOP) { set_err("ENDLOOP without LOOP", pc); goto bad; }
            P->match[stk[sp - 1]] = (int32_t)pc;
            P->match[pc] = stk[sp - 1];
            sp--;
        } else if (op == B_OBS) {
            uint32_t ns = (uint32_t)w_a(P, pc);
            if (pc + ns >= P->n_instr) { set_err("OBS strides run past the end", pc); goto bad; }
            for (uint32_t d = 1; d <= ns; ++d)
                if (w_op(P, pc + d) != B_OBSX) { set_err("missing OBSX word", pc); goto bad; }
            for (uint32_t d = 1; d <= ns; ++d) P->match[pc + d] = -1;
            pc += ns;
        } else if (op == B_LOADL || op == B_STOREL) {
            if ((int)w_imm(P, pc) > maxloc) maxloc = (int)w_imm(P, pc);
        }
    }
    if (sp != 0) { set_err("unterminated block", -1); goto bad; }
    P->n_locals = maxloc + 1;
    free(stk);
    return 0;
bad:
    free(stk);
    free(P->match);
    P->match = NULL;
    return -1;
}

/* ---------------- per-lane state ---------------- */
typedef struct {
    Node *nodes;
    int n_nodes, cap_nodes;
    int *stack;
    int sp, cap_stack;
    int *locals;
    Val *adj;
    int cap_adj;
    int *packbuf;       /* arena for PACK input lists */
    int n_pack, cap_pack;
} Lane;

static int new_node(Lane *S) {
    if (S->n_nodes == S->cap_nodes) {
        int nc = S->cap_nodes ? 2 * S->cap_nodes : 1024;
        Node *nn = (Node *)realloc(S->nodes, sizeof(Node) * (size_t)nc);
        if (!nn) return -1;
        S->nodes = nn;
        S->cap_nodes = nc;
    }
    Node *x = &S->nodes[S->n_nodes];
    x->kind = K_LEAF;
    x->in[0] = x->in[1] = -1;
    x->npack = 0;
    x->pack_in = NULL;
    x->aux = 0;
    return S->n_nodes++;
}

static int push(Lane *S, int id) {
    if (S->sp == S->cap_stack) {
        int nc = S->cap_stack ? 2 * S->cap_stack : 64;
        int *ns = (int *)realloc(S->stack, sizeof(int) * (size_t)nc);
        if (!ns) return -1;
        S->stack = ns;
        S->cap_stack = nc;
    }
    S->stack[S->sp++] = id;
    return 0;
}

static int is_scalar(const Val *v) { return v->rows == 1 && v->cols == 1; }
static int nel(const Val *v) { return v->rows * v->cols; }
static real clampv(real x) { return x < CLAMP_EPS ? CLAMP_EPS : x; }

/* Optional perturbation of library transcendental results (exp, log, sin,
 * cos, pow; forward values and those inside adjoint rules) by a
 * pseudo-random whole number of units in the last place in [-ulps, ulps],
 * drawn per evaluation from a counter-based hash of (seed, lane, count).
 * Another correct math library differs from this one's results by about that
 * much, so the spread of a lane's result over a few seeds measures how
 * strongly library last-ulp differences move it (its conditioning with
 * respect to transcendental rounding).  Off (ulps = 0) by default. */
typedef struct { int ulps; uint64_t key, count; } Perturb;
static __thread Perturb g_pt;

static uint64_t mix64(uint64_t z) {     /* splitmix64 finaliser (Steele, Lea, Flood 2014) */
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static real tr(real y) {
    if (g_pt.ulps <= 0 || !(y == y) || y - y != 0) return y;
    uint64_t h = mix64(g_pt.key ^ mix64(g_pt.count++));
    int d = (int)(h % (uint64_t)(2 * g_pt.ulps + 1)) - g_pt.ulps;
#ifdef ORACLE_LONG_DOUBLE
    for (; d > 0; --d) y = nextafterl(y, (real)INFINITY);
    for (; d < 0; ++d) y = nextafterl(y, -(real)INFINITY);
#else
    for (; d > 0; --d) y = nextafter(y, INFINITY);
    for (; d < 0; ++d) y = nextafter(y, -INFINITY);
#endif
    return y;
}

/* Z = X Y with an fma chain over the inner index, ascending. */
static void matmul(const Val *X, const Val *Y, Val *Z) {
    int m = X->rows, k = X->cols, n = Y->cols;
    Z->rows = m;
    Z->cols = n;
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < n; ++j) {
            real t = X->e[i * k + 0] * Y->e[0 * n + j];
            for (int p = 1; p < k; ++p) t = R_FMA(X->e[i * k + p], Y->e[p * n + j], t);
            Z->e[i * n + j] = t;
        }
}

static void transpose(const Val *X, Val *Z) {
    Z->rows = X->cols;
    Z->cols = X->rows;
    for (int i = 0; i < X->rows; ++i)
        for (int j = 0; j < X->cols; ++j) Z->e[j * X->rows + i] = X->e[i * X->cols + j];
}

/* det = a*d - b*c for 2x2, the element itself for 1x1 */
static real det_of(const Val *A) {
    if (A->rows == 1) return A->e[0];
    real t1 = A->e[0] * A->e[3];
    real t2 = A->e[1] * A->e[2];
    return t1 - t2;
}

/* inverse of a 1x1 or 2x2 matrix: adjugate times r = 1/det */
static void inverse(const Val *A, Val *B) {
    B->rows = A->rows;
    B->cols = A->cols;
    if (A->rows == 1) {
        B->e[0] = (real)1 / A->e[0];
        return;
    }
    real r = (real)1 / det_of(A);
    B->e[0] = A->e[3] * r;
    B->e[1] = (-A->e[1]) * r;
    B->e[2] = (-A->e[2]) * r;
    B->e[3] = A->e[0] * r;
}

static int shape_ok_small_square(const Val *A) {
    return A->rows == A->cols && (A->rows == 1 || A->rows == 2);
}

/* Evaluate one numeric primitive; returns 0 or -1 (shape error). */
static int forward_op(int op, const Val *a, const Val *b, Val *z) {
    int n;
    switch (op) {
    case B_ADD:
    case B_SUB:
        if (a->rows != b->rows || a->cols != b->cols) return -1;
        *z = *a;
        for (int i = 0; i < nel(a); ++i) z->e[i] = op == B_ADD ? a->e[i] + b->e[i] : a->e[i] - b->e[i];
        return 0;
    case B_MUL:
        if (a->rows == b->rows && a->cols == b->cols) {
            *z = *a;
            for (int i = 0; i < nel(a); ++i) z->e[i] = a->e[i] * b->e[i];
        } else if (is_scalar(a)) {
            *z = *b;
            for (int i = 0; i < nel(b); ++i) z->e[i] = a->e[0] * b->e[i];
        } else if (is_scalar(b)) {
            *z = *a;
            for (int i = 0; i < nel(a); ++i) z->e[i] = a->e[i] * b->e[0];
        } else {
            return -1;
        }
        return 0;
    case B_DIV:
        if (a->rows == b->rows && a->cols == b->cols) {
            *z = *a;
            for (int i = 0; i < nel(a); ++i) z->e[i] = a->e[i] / b->e[i];
        } else if (is_scalar(b)) {
            *z = *a;
            for (int i = 0; i < nel(a); ++i) z->e[i] = a->e[i] / b->e[0];
        } else {
            return -1;
        }
        return 0;
    case B_NEG: case B_EXP: case B_LOG: case B_SQRT: case B_SIN: case B_COS: case B_ABS:
        *z = *a;
        for (int i = 0; i < nel(a); ++i) {
            real x = a->e[i];
            switch (op) {
            case B_NEG: z->e[i] = -x; break;
            case B_EXP: z->e[i] = tr(R_EXP(x)); break;
            case B_LOG: z->e[i] = tr(R_LOG(clampv(x))); break;
            case B_SQRT: z->e[i] = R_SQRT(clampv(x)); break;
            case B_SIN: z->e[i] = tr(R_SIN(x)); break;
            case B_COS: z->e[i] = tr(R_COS(x)); break;
            default: z->e[i] = R_FABS(x); break;
            }
        }
        return 0;
    case B_POW:
        if (!is_scalar(a) || !is_scalar(b)) return -1;
        z->rows = z->cols = 1;
        z->e[0] = tr(R_POW(a->e[0], b->e[0]));
        return 0;
    case B_DOT:
        if (a->rows != b->rows || a->cols != b->cols) return -1;
        n = nel(a);
        z->rows = z->cols = 1;
        z->e[0] = a->e[0] * b->e[0];
        for (int i = 1; i < n; ++i) z->e[0] = R_FMA(a->e[i], b->e[i], z->e[0]);
        return 0;
    case B_MATMUL:
        if (a->cols != b->rows) return -1;
        matmul(a, b, z);
        return 0;
    case B_TRANSPOSE:
        transpose(a, z);
        return 0;
    case B_TRACE:
        if (a->rows != a->cols) return -1;
        z->rows = z->cols = 1;
        z->e[0] = a->e[0];
        for (int i = 1; i < a->rows; ++i) z->e[0] = z->e[0] + a->e[i * a->cols + i];
        return 0;
    case B_INV:
        if (!shape_ok_small_square(a)) return -1;
        inverse(a, z);
        return 0;
    case B_DET:
        if (!shape_ok_small_square(a)) return -1;
        z->rows = z->cols = 1;
        z->e[0] = det_of(a);
        return 0;
    case B_LOGDET:
        if (!shape_ok_small_square(a)) return -1;
        z->rows = z->cols = 1;
        z->e[0] = tr(R_LOG(clampv(det_of(a))));
        return 0;
    case B_OUTER:
        if (a->cols != 1 || b->cols != 1) return -1;
        z->rows = a->rows;
        z->cols = b->rows;
        for (int i = 0; i < a->rows; ++i)
            for (int j = 0; j < b->rows; ++j) z->e[i * b->rows + j] = a->e[i] * b->e[j];
        return 0;
    }
    return -1;
}

static int arity(int op) {
    switch (op) {
    case B_ADD: case B_SUB: case B_MUL: case B_DIV: case B_POW: case B_DOT:
    case B_MATMUL: case B_OUTER:
        return 2;
    case B_NEG: case B_EXP: case B_LOG: case B_SQRT: case B_SIN: case B_COS:
    case B_ABS: case B_TRANSPOSE: case B_TRACE: case B_INV: case B_DET: case B_LOGDET:
        return 1;
    }
    return -1;
}

/* Run one lane forward; returns 0 and the loss node id in *loss_id. */
/* Branch bookkeeping of one lane's walk: numeric IFLTs are counted in the
 * order the walk meets them (a loop body's IFLT counts once per trip). */
#define MAX_TIES 8
typedef struct {
    real margin;       /* smallest relative gap |a-b|/max(|a|,|b|) met so far */
    int64_t seen;      /* encounters so far */
    int64_t flip;      /* encounter whose decision is inverted (-1: none) */
    real tie_tol;      /* gaps at or below this are recorded as near ties */
    int n_ties;        /* recorded near ties, closest first */
    int64_t tie_at[MAX_TIES];
    real tie_m[MAX_TIES];
} Branches;

/* keep the MAX_TIES smallest gaps at or below tie_tol, in ascending order
 * (equal gaps in the order met) */
static void note_tie(Branches *br, real m, int64_t at) {
    if (!(m <= br->tie_tol)) return;
    int k = br->n_ties < MAX_TIES ? br->n_ties++ : MAX_TIES;
    if (k == MAX_TIES) {
        if (!(m < br->tie_m[MAX_TIES - 1])) return;
        k = MAX_TIES - 1;
    }
    while (k > 0 && m < br->tie_m[k - 1]) {
        br->tie_m[k] = br->tie_m[k - 1];
        br->tie_at[k] = br->tie_at[k - 1];
        --k;
    }
    br->tie_m[k] = m;
    br->tie_at[k] = at;
}

static int run_forward(const Prog *P, Lane *S, const real *theta, const double *obs,
                       int *loss_id, Branches *br) {
    S->n_nodes = 0;
    S->sp = 0;
    S->n_pack = 0;
    for (int j = 0; j < P->n_locals; ++j) S->locals[j] = -1;
    for (uint32_t i = 0; i < P->n_params; ++i) {
        int id = new_node(S);
        if (id < 0) return E_NOMEM;
        S->nodes[id].kind = K_PARAM;
        S->nodes[id].aux = (int)i;
        S->nodes[id].v.rows = S->nodes[id].v.cols = 1;
        S->nodes[id].v.e[0] = theta[i];
    }
    int lp_pc[64], lp_n[64], lp_k[64], ld = 0;  /* loop frames */
    int pc = 0;
    for (;;) {
        if (pc < 0 || (uint32_t)pc >= P->n_instr) { set_err("fell off the program", pc); return E_RUNTIME; }
        int op = w_op(P, pc);
        uint32_t imm = w_imm(P, pc);
        switch (op) {
        case B_HALT: {
            if (S->sp != 1 || !is_scalar(&S->nodes[S->stack[0]].v)) { set_err("HALT needs one scalar", pc); return E_RUNTIME; }
            *loss_id = S->stack[0];
            return OK;
        }
        case B_PUSH: case B_OBS: {
            double val;
            if (op == B_PUSH) {
                if (imm >= P->n_consts) { set_err("bad const index", pc); return E_RUNTIME; }
                val = P->consts[imm];
            } else {
                int ns = w_a(P, pc);
                int64_t idx = (int64_t)imm;
                if (ns > ld) { set_err("OBS stride beyond loop depth", pc); return E_RUNTIME; }
                for (int d = 0; d < ns; ++d) idx += (int64_t)(int32_t)w_imm(P, pc + 1 + d) * lp_k[ld - 1 - d];
                if (idx < 0 || idx >= (int64_t)P->n_obs) { set_err("obs index out of range", pc); return E_RUNTIME; }
                val = obs[idx];
                pc += ns;
            }
            int id = new_node(S);
            if (id < 0) return E_NOMEM;
            S->nodes[id].kind = K_LEAF;
            S->nodes[id].v.rows = S->nodes[id].v.cols = 1;
            S->nodes[id].v.e[0] = (real)val;
            if (push(S, id)) return E_NOMEM;
            break;
        }
        case B_PARAM:
            if (imm >= P->n_params) { set_err("bad param index", pc); return E_RUNTIME; }
            if (push(S, (int)imm)) return E_NOMEM;
            break;
        case B_LOADL:
            if ((int)imm >= P->n_locals || S->locals[imm] < 0) { set_err("unset local", pc); return E_RUNTIME; }
            if (push(S, S->locals[imm])) return E_NOMEM;
            break;
        case B_STOREL:
            if (S->sp < 1) { set_err("stack underflow", pc); return E_RUNTIME; }
            S->locals[imm] = S->stack[--S->sp];
            break;
        case B_DUP:
            if (S->sp < 1) { set_err("stack underflow", pc); return E_RUNTIME; }
            if (push(S, S->stack[S->sp - 1])) return E_NOMEM;
            break;
        case B_OVER:
            if (S->sp < 2) { set_err("stack underflow", pc); return E_RUNTIME; }
            if (push(S, S->stack[S->sp - 2])) return E_NOMEM;
            break;
        case B_SWAP: {
            if (S->sp < 2) { set_err("stack underflow", pc); return E_RUNTIME; }
            int t = S->stack[S->sp - 1];
            S->stack[S->sp - 1] = S->stack[S->sp - 2];
            S->stack[S->sp - 2] = t;
            break;
        }
        case B_DROP:
            if (S->sp < 1) { set_err("stack underflow", pc); return E_RUNTIME; }
            S->sp--;
            break;
        case B_PACK: {
            int r = w_a(P, pc), c = w_b(P, pc), n = r * c;
            if (r < 1 || c < 1 || r > 4 || c > 4) { set_err("bad PACK shape", pc); return E_RUNTIME; }
            if (S->sp < n) { set_err("stack underflow", pc); return E_RUNTIME; }
            if (S->n_pack + n > S->cap_pack) {
                /* the arena only grows; node pack_in pointers are offsets resolved below */
                int nc = S->cap_pack ? 2 * S->cap_pack : 1024;
                while (nc < S->n_pack + n) nc *= 2;
                int *nb = (int *)realloc(S->packbuf, sizeof(int) * (size_t)nc);
                if (!nb) return E_NOMEM;
                S->packbuf = nb;
                S->cap_pack = nc;
            }
            int id = new_node(S);
            if (id < 0) return E_NOMEM;
            Node *x = &S->nodes[id];
            x->kind = B_PACK;
            x->npack = n;
            x->aux = S->n_pack;   /* offset into packbuf */
            x->v.rows = r;
            x->v.cols = c;
            for (int i = 0; i < n; ++i) {
                int src = S->stack[S->sp - n + i];
                if (!is_scalar(&S->nodes[src].v)) { set_err("PACK of a non-scalar", pc); return E_RUNTIME; }
                S->packbuf[S->n_pack + i] = src;
                x->v.e[i] = S->nodes[src].v.e[0];
            }
            S->n_pack += n;
            S->sp -= n;
            if (push(S, id)) return E_NOMEM;
            break;
        }
        case B_INDEX: {
            if (S->sp < 1) { set_err("stack underflow", pc); return E_RUNTIME; }
            int src = S->stack[S->sp - 1];
            int i = w_a(P, pc), j = w_b(P, pc);
            const Val *A = &S->nodes[src].v;
            if (i >= A->rows || j >= A->cols) { set_err("INDEX out of range", pc); return E_RUNTIME; }
            int id = new_node(S);
            if (id < 0) return E_NOMEM;
            Node *x = &S->nodes[id];
            x->kind = B_INDEX;
            x->in[0] = src;
            x->aux = i * S->nodes[src].v.cols + j;
            x->v.rows = x->v.cols = 1;
            x->v.e[0] = S->nodes[src].v.e[x->aux];
            S->stack[S->sp - 1] = id;
            break;
        }
        case B_LOOP:
            if (imm == 0) { pc = P->match[pc] + 1; continue; }
            if (ld == 64) { set_err("loop nesting too deep", pc); return E_RUNTIME; }
            lp_pc[ld] = pc + 1;
            lp_n[ld] = (int)imm;
            lp_k[ld] = 0;
            ld++;
            break;
        case B_ENDLOOP:
            if (ld == 0) { set_err("ENDLOOP outside a loop", pc); return E_RUNTIME; }
            if (++lp_k[ld - 1] < lp_n[ld - 1]) { pc = lp_pc[ld - 1]; continue; }
            ld--;
            break;
        case B_IFLT: {
            if (S->sp < 2) { set_err("stack underflow", pc); return E_RUNTIME; }
            int bi = S->stack[--S->sp], ai = S->stack[--S->sp];
            if (!is_scalar(&S->nodes[ai].v) || !is_scalar(&S->nodes[bi].v)) { set_err("IFLT on a non-scalar", pc); return E_RUNTIME; }
            real a = S->nodes[ai].v.e[0], b = S->nodes[bi].v.e[0];
            int take_then = a < b;
            if (br) {
                real den = R_FABS(a) > R_FABS(b) ? R_FABS(a) : R_FABS(b);
                real m = den > 0 ? R_FABS(a - b) / den : 0;
                if (a != a || b != b) m = 0;
                if (m < br->margin) br->margin = m;
                note_tie(br, m, br->seen);
                /* the other arm of an encounter whose operands sit within
                 * rounding of a tie is the realized trace of an equally
                 * valid evaluation (Property 1: exact on either path) */
                if (br->seen == br->flip) take_then = !take_then;
                br->seen++;
            }
            if (take_then) break;             /* then-arm follows */
            pc = P->match[pc] + 1;            /* first word after ELSE */
            continue;
        }
        case B_ELSE:                          /* end of a taken then-arm */
            pc = P->match[pc] + 1;
            continue;
        case B_ENDIF:
            break;
        case B_OBSX:
            set_err("stray OBSX word", pc);
            return E_RUNTIME;
        default: {
            int ar = arity(op);
            if (ar < 0) { set_err("unknown opcode", pc); return E_BYTECODE; }
            if (S->sp < ar) { set_err("stack underflow", pc); return E_RUNTIME; }
            int bi = ar == 2 ? S->stack[S->sp - 1] : -1;
            int ai = S->stack[S->sp - ar];
            int id = new_node(S);
            if (id < 0) return E_NOMEM;
            Node *x = &S->nodes[id];
            x->kind = op;
            x->in[0] = ai;
            x->in[1] = bi;
            if (forward_op(op, &S->nodes[ai].v, bi >= 0 ? &S->nodes[bi].v : NULL, &x->v)) {
                set_err("shape error", pc);
                return E_RUNTIME;
            }
            S->sp -= ar;
            if (push(S, id)) return E_NOMEM;
            break;
        }
        }
        pc++;
    }
}

static int all_zero(const Val *g) {
    for (int i = 0; i < nel(g); ++i)
        if (g->e[i] != 0) return 0;
    return 1;
}

/* Reverse sweep over the realized node list (table tab:adjoints). */
static void run_reverse(const Prog *P, Lane *S, int loss_id) {
    (void)P;
    for (int k = 0; k < S->n_nodes; ++k) {
        S->adj[k].rows = S->nodes[k].v.rows;
        S->adj[k].cols = S->nodes[k].v.cols;
        for (int i = 0; i < MAXE; ++i) S->adj[k].e[i] = 0;
    }
    S->adj[loss_id].e[0] = 1;
    for (int k = S->n_nodes - 1; k >= 0; --k) {
        Node *x = &S->nodes[k];
        if (x->kind == K_PARAM || x->kind == K_LEAF) continue;
        const Val *g = &S->adj[k];
        if (all_zero(g)) continue;
        const Val *z = &x->v;
        const Val *a = x->in[0] >= 0 ? &S->nodes[x->in[0]].v : NULL;
        const Val *b = x->in[1] >= 0 ? &S->nodes[x->in[1]].v : NULL;
        Val *ga = x->in[0] >= 0 ? &S->adj[x->in[0]] : NULL;
        Val *gb = x->in[1] >= 0 ? &S->adj[x->in[1]] : NULL;
        int n = nel(z);
        switch (x->kind) {
        case B_ADD:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i];
            for (int i = 0; i < n; ++i) gb->e[i] = gb->e[i] + g->e[i];
            break;
        case B_SUB:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i];
            for (int i = 0; i < n; ++i) gb->e[i] = gb->e[i] - g->e[i];
            break;
        case B_MUL:
            if (a->rows == b->rows && a->cols == b->cols) {
                for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] * b->e[i];
                for (int i = 0; i < n; ++i) gb->e[i] = gb->e[i] + g->e[i] * a->e[i];
            } else if (is_scalar(a)) {        /* z = s * M */
                real t = g->e[0] * b->e[0];
                for (int i = 1; i < n; ++i) t = R_FMA(g->e[i], b->e[i], t);
                ga->e[0] = ga->e[0] + t;
                for (int i = 0; i < n; ++i) gb->e[i] = gb->e[i] + g->e[i] * a->e[0];
            } else {                          /* z = M * s */
                for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] * b->e[0];
                real t = g->e[0] * a->e[0];
                for (int i = 1; i < n; ++i) t = R_FMA(g->e[i], a->e[i], t);
                gb->e[0] = gb->e[0] + t;
            }
            break;
        case B_DIV:
            if (a->rows == b->rows && a->cols == b->cols) {
                for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] / b->e[i];
                for (int i = 0; i < n; ++i) gb->e[i] = gb->e[i] - (g->e[i] * z->e[i]) / b->e[i];
            } else {                          /* z = M / s */
                for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] / b->e[0];
                real t = g->e[0] * z->e[0];
                for (int i = 1; i < n; ++i) t = R_FMA(g->e[i], z->e[i], t);
                gb->e[0] = gb->e[0] - t / b->e[0];
            }
            break;
        case B_NEG:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] - g->e[i];
            break;
        case B_EXP:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] * z->e[i];
            break;
        case B_LOG:
            for (int i = 0; i < n; ++i)
                if (a->e[i] > CLAMP_EPS) ga->e[i] = ga->e[i] + g->e[i] / a->e[i];
            break;
        case B_SQRT:
            for (int i = 0; i < n; ++i)
                if (a->e[i] > CLAMP_EPS) ga->e[i] = ga->e[i] + g->e[i] / ((real)2 * z->e[i]);
            break;
        case B_SIN:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] + g->e[i] * tr(R_COS(a->e[i]));
            break;
        case B_COS:
            for (int i = 0; i < n; ++i) ga->e[i] = ga->e[i] - g->e[i] * tr(R_SIN(a->e[i]));
            break;
        case B_ABS:
            for (int i = 0; i < n; ++i) {
                real s = a->e[i] > 0 ? g->e[i] : (a->e[i] < 0 ? -g->e[i] : (real)0);
                ga->e[i] = ga->e[i] + s;
            }
            break;
        case B_POW:
            ga->e[0] = ga->e[0] + ((g->e[0] * b->e[0]) * z->e[0]) / a->e[0];
            gb->e[0] = gb->e[0] + (g->e[0] * z->e[0]) * tr(R_LOG(a->e[0]));
            break;
        case B_DOT: {
            int m = nel(a);
            for (int i = 0; i < m; ++i) ga->e[i] = ga->e[i] + g->e[0] * b->e[i];
            for (int i = 0; i < m; ++i) gb->e[i] = gb->e[i] + g->e[0] * a->e[i];
            break;
        }
        case B_MATMUL: {
            Val bt, at, da, db;
            transpose(b, &bt);
            transpose(a, &at);
            matmul(g, &bt, &da);      /* dA = g B^T */
            matmul(&at, g, &db);      /* dB = A^T g */
            for (int i = 0; i < nel(a); ++i) ga->e[i] = ga->e[i] + da.e[i];
            for (int i = 0; i < nel(b); ++i) gb->e[i] = gb->e[i] + db.e[i];
            break;
        }
        case B_TRANSPOSE: {
            Val gt;
            transpose(g, &gt);
            for (int i = 0; i < nel(a); ++i) ga->e[i] = ga->e[i] + gt.e[i];
            break;
        }
        case B_TRACE:
            for (int i = 0; i < a->rows; ++i) ga->e[i * a->cols + i] = ga->e[i * a->cols + i] + g->e[0];
            break;
        case B_INV: {
            Val bt, m1, m2;
            transpose(z, &bt);
            matmul(&bt, g, &m1);      /* B^T g */
            matmul(&m1, &bt, &m2);    /* (B^T g) B^T */
            for (int i = 0; i < nel(a); ++i) ga->e[i] = ga->e[i] - m2.e[i];
            break;
        }
        case B_DET: {
            Val ai;
            inverse(a, &ai);
            real gz = g->e[0] * z->e[0];
            int r = a->rows;
            for (int i = 0; i < r; ++i)
                for (int j = 0; j < r; ++j) ga->e[i * r + j] = ga->e[i * r + j] + gz * ai.e[j * r + i];
            break;
        }
        case B_LOGDET: {
            if (!(det_of(a) > CLAMP_EPS)) break;
            Val ai;
            inverse(a, &ai);
            int r = a->rows;
            for (int i = 0; i < r; ++i)
                for (int j = 0; j < r; ++j) ga->e[i * r + j] = ga->e[i * r + j] + g->e[0] * ai.e[j * r + i];
            break;
        }
        case B_OUTER: {
            int m = a->rows, q = b->rows;
            for (int i = 0; i < m; ++i) {
                real t = g->e[i * q + 0] * b->e[0];
                for (int j = 1; j < q; ++j) t = R_FMA(g->e[i * q + j], b->e[j], t);
                ga->e[i] = ga->e[i] + t;
            }
            for (int j = 0; j < q; ++j) {
                real t = g->e[0 * q + j] * a->e[0];
                for (int i = 1; i < m; ++i) t = R_FMA(g->e[i * q + j], a->e[i], t);
                gb->e[j] = gb->e[j] + t;
            }
            break;
        }
        case B_PACK:
            for (int i = 0; i < x->npack; ++i) {
                Val *gs = &S->adj[S->packbuf[x->aux + i]];
                gs->e[0] = gs->e[0] + g->e[i];
            }
            break;
        case B_INDEX:
            ga->e[x->aux] = ga->e[x->aux] + g->e[0];
            break;
        }
    }
}

typedef struct {
    const Prog *P;
    const double *params, *obs;
    int64_t ld_p, ld_g, l0, l1;
    double *loss, *grad, *margin;
    int64_t *ties;
    double tie_tol;
    const int64_t *flip;
    uint64_t perturb_seed;
    int perturb_ulps;
    int status;
} Job;

static void *worker(void *arg) {
    Job *J = (Job *)arg;
    const Prog *P = J->P;
    Lane S;
    memset(&S, 0, sizeof S);
    S.locals = (int *)malloc(sizeof(int) * (size_t)(P->n_locals > 0 ? P->n_locals : 1));
    real *theta = (real *)malloc(sizeof(real) * (P->n_params + 1));
    J->status = OK;
    for (int64_t l = J->l0; l < J->l1; ++l) {
        for (uint32_t i = 0; i < P->n_params; ++i) theta[i] = (real)J->params[l * J->ld_p + i];
        int loss_id = -1;
        Branches br;
        memset(&br, 0, sizeof br);
        br.margin = (real)INFINITY;
        br.flip = J->flip ? J->flip[l] : -1;
        br.tie_tol = (real)J->tie_tol;
        g_pt.ulps = J->perturb_ulps;
        g_pt.key = mix64(J->perturb_seed) ^ (uint64_t)l;
        g_pt.count = 0;
        int st = run_forward(P, &S, theta, J->obs, &loss_id, &br);
        if (st != OK) { J->status = st; break; }
        J->loss[l] = (double)S.nodes[loss_id].v.e[0];
        if (J->margin) J->margin[l] = (double)br.margin;
        if (J->ties)
            for (int k = 0; k < MAX_TIES; ++k) J->ties[l * MAX_TIES + k] = k < br.n_ties ? br.tie_at[k] : -1;
        if (J->grad) {
            if (S.cap_adj < S.n_nodes) {
                free(S.adj);
                S.adj = (Val *)malloc(sizeof(Val) * (size_t)S.n_nodes);
                if (!S.adj) { J->status = E_NOMEM; break; }
                S.cap_adj = S.n_nodes;
            }
            run_reverse(P, &S, loss_id);
            for (uint32_t i = 0; i < P->n_params; ++i) J->grad[l * J->ld_g + i] = (double)S.adj[i].e[0];
        }
    }
    free(S.nodes);
    free(S.stack);
    free(S.locals);
    free(S.adj);
    free(S.packbuf);
    free(theta);
    return NULL;
}

/*
 * Evaluate loss[L] (and grad[L, n_params] when grad != NULL) for L lanes.
 * params: lane l, parameter i at params[l*ld_p + i]; grad likewise with ld_g.
 * margin (optional): per lane, the smallest relative gap |a-b|/max(|a|,|b|)
 * seen at any IFLT, +inf when the lane meets none.
 * ties (optional, [L, 8]): per lane, the encounters (IFLTs counted from 0 in
 * the order the lane's walk meets them) whose gap is at most tie_tol, the 8
 * smallest gaps in ascending order, -1 padded.
 * flip (optional): per lane, one encounter whose decision is inverted (-1:
 * none): the lane's realized trace had that comparison gone the other way.
 * Used to judge lanes whose comparison is a near tie.
 * perturb_ulps > 0: every library transcendental result is moved by a
 * pseudo-random whole number of ulps in [-perturb_ulps, perturb_ulps]
 * (counter-based hash of perturb_seed, the lane and the evaluation count);
 * used to measure a lane's sensitivity to math-library rounding.
 * Lanes are split into nthreads contiguous blocks; results do not depend on
 * the thread count.  Returns 0, or an error code with a message in
 * ndvm_oracle_error().
 */
int ENTRY(ndvm_oracle_run)(const uint8_t *bc, size_t bc_len, const double *params, int64_t L,
                           int64_t ld_p, const double *obs, int64_t n_obs, double *loss,
                           double *grad, int64_t ld_g, double *margin, int64_t *ties,
                           double tie_tol, const int64_t *flip, uint64_t perturb_seed,
                           int perturb_ulps, int nthreads) {
    Prog P;
    if (!bc || L < 0 || !loss || (L > 0 && !params)) { set_err("bad arguments", -1); return E_ARG; }
    if (parse(bc, bc_len, &P)) return E_BYTECODE;
    if ((int64_t)P.n_obs != n_obs || (P.n_obs > 0 && !obs) || ld_p < (int64_t)P.n_params ||
        (grad && ld_g < (int64_t)P.n_params)) {
        free(P.match);
        set_err("argument sizes do not match the program", -1);
        return E_ARG;
    }
    if (nthreads < 1) nthreads = 1;
    if (nthreads > L && L > 0) nthreads = (int)L;
    if (L == 0) { free(P.match); return OK; }
    Job *jobs = (Job *)calloc((size_t)nthreads, sizeof(Job));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = (Job){&P, params, obs, ld_p, ld_g, L * t / nthreads, L * (t + 1) / nthreads,
                        loss, grad, margin, ties, tie_tol, flip, perturb_seed, perturb_ulps, OK};
        pthread_create(&th[t], NULL, worker, &jobs[t]);
    }
    int st = OK;
    for (int t = 0; t < nthreads; ++t) {
        pthread_join(th[t], NULL);
        if (jobs[t].status != OK && st == OK) st = jobs[t].status;
    }
    free(jobs);
    free(th);
    free(P.match);
    return st;
}
