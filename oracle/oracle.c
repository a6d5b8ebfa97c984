/*
 * CPU oracle for the distributed deep Q-learning hot path (arXiv 1508.04186).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant with the HIP library, and the HIP library never
 * calls it.
 *
 * Plain, slow, obviously correct: direct nested loops, every floating-point
 * operation in double precision.  Parameters come in as double (the callers
 * widen the same float32 arrays the GPU receives); optimizer state is rounded
 * to float32 only where the GPU stores float32.  Samples are processed in
 * parallel (OpenMP), but every reduction over samples is a sequential sum in
 * sample order, so results do not depend on the thread count.
 *
 * What it computes, by passage of the paper:
 *   oracle_replay_gather   uniform minibatch draw from the replay memory
 *                          (Sec. III.C; Alg. 1 "uniformly sample"): the
 *                          transition of record i is (phi_i, a_i, r_i, phi_{i+1}).
 *   oracle_forward_q       Q(phi; theta), one output per action (Sec. III.A):
 *                          valid-padding convolutions with ReLU f(x)=max(0,x),
 *                          a hidden fully connected layer with ReLU, and a
 *                          linear output layer.  Input bytes are scaled by 1/255.
 *   oracle_select_actions  greedy action argmax_a Q (Sec. II.A) with
 *                          epsilon-greedy exploration (Sec. III.B; Alg. 1).
 *   oracle_td_gradient     targets y_j = r_j (terminal) or r_j + gamma max_a'
 *                          Q(phi_{j+1}, a'; theta^-) and the gradient of
 *                          (1/b) sum_j 1/2 (Q(phi_j, a_j; theta) - y_j)^2
 *                          (Alg. 1; Eq. (1)), with y held constant.
 *   oracle_apply_update    the parameter-server update: plain gradient
 *                          descent (Sec. III.B), the RMSProp rule of Alg. 2,
 *                          and AdaGrad (named in Sec. IV.D.2).
 *
 *   oracle_snake_*         the actor side of Alg. 1: the Snake game of
 *                          Sec. V.A stepped by a chosen action, rendered as
 *                          stacked 84x84 frames, and the experiences stored
 *                          in a replay memory that keeps the last N of them
 *                          (Sec. III.C), pooled over game instances.
 *   oracle_preprocess      phi (Sec. III.A, Fig. 2): raw RGB screens
 *                          gray-scaled, cropped and down-sampled to 84x84.
 *
 * The bf16-input variant (net->bf16_inputs = 1) computes the same functions
 * with every operand of the layer contractions -- the conv and fc1 weights,
 * the conv and fc1 input activations, and the back-propagated gradients
 * that multiply weights or activations -- first rounded to float32 (the
 * precision in which they are stored) and then to bfloat16 with round to
 * nearest, ties to even; products and sums stay in double.  The input bytes
 * are exact in bfloat16, and the 1/255 scale applies after the sum.  Bias
 * gradients, the fc2 output layer and the ReLU decisions use the unrounded
 * values.
 *
 * Readings where the paper is silent or garbled are stated at each function.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC oracle.c -o liboracle.so
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define ORACLE_MAX_CONV 3

typedef struct {
    int32_t in_c, in_h, in_w;
    int32_t n_conv;
    int32_t conv_out[ORACLE_MAX_CONV];
    int32_t conv_k[ORACLE_MAX_CONV];
    int32_t conv_stride[ORACLE_MAX_CONV];
    int32_t fc_hidden, n_actions;
    int32_t bf16_inputs;   /* 1: the bf16-input variant described above */
} oracle_net;

enum { ORACLE_OK = 0, ORACLE_EINVAL = -1, ORACLE_ERANGE = -2, ORACLE_ENOMEM = -3 };
enum { RULE_SGD = 0, RULE_RMSPROP = 1, RULE_ADAGRAD = 2 };

/* ------------------------------------------------------------------------ */
/* Shapes and the flat parameter layout: for each conv layer W[out][in][k][k]
 * then b[out]; then fc1 W[hidden][flat] and b[hidden]; then fc2
 * W[actions][hidden] and b[actions].  The fc1 input is the last conv output
 * flattened channel-major (c, y, x). */

typedef struct {
    int c[ORACLE_MAX_CONV + 1], h[ORACLE_MAX_CONV + 1], w[ORACLE_MAX_CONV + 1];
    int64_t w_off[ORACLE_MAX_CONV + 2], b_off[ORACLE_MAX_CONV + 2];
    int64_t flat, n_params;
    int64_t max_act; /* largest activation of one sample */
} shapes_t;

static int make_shapes(const oracle_net* net, shapes_t* sh) {
    if (!net || net->n_conv < 0 || net->n_conv > ORACLE_MAX_CONV) return ORACLE_EINVAL;
    if (net->in_c <= 0 || net->in_h <= 0 || net->in_w <= 0) return ORACLE_EINVAL;
    if (net->fc_hidden <= 0 || net->n_actions <= 0) return ORACLE_EINVAL;
    sh->c[0] = net->in_c; sh->h[0] = net->in_h; sh->w[0] = net->in_w;
    int64_t off = 0, mx = (int64_t)net->in_c * net->in_h * net->in_w;
    for (int l = 0; l < net->n_conv; ++l) {
        int k = net->conv_k[l], s = net->conv_stride[l], o = net->conv_out[l];
        if (k <= 0 || s <= 0 || o <= 0 || sh->h[l] < k || sh->w[l] < k) return ORACLE_EINVAL;
        sh->c[l + 1] = o;
        sh->h[l + 1] = (sh->h[l] - k) / s + 1;
        sh->w[l + 1] = (sh->w[l] - k) / s + 1;
        sh->w_off[l] = off; off += (int64_t)o * sh->c[l] * k * k;
        sh->b_off[l] = off; off += o;
        int64_t a = (int64_t)o * sh->h[l + 1] * sh->w[l + 1];
        if (a > mx) mx = a;
    }
    int L = net->n_conv;
    sh->flat = (int64_t)sh->c[L] * sh->h[L] * sh->w[L];
    sh->w_off[L] = off; off += (int64_t)net->fc_hidden * sh->flat;
    sh->b_off[L] = off; off += net->fc_hidden;
    sh->w_off[L + 1] = off; off += (int64_t)net->n_actions * net->fc_hidden;
    sh->b_off[L + 1] = off; off += net->n_actions;
    sh->n_params = off;
    if (net->fc_hidden > mx) mx = net->fc_hidden;
    sh->max_act = mx;
    return ORACLE_OK;
}

/* out[i] = the bf16 contraction operand of in[i] (bf16_round below), so the
 * tests can check the rounding itself. */
static double bf16_round(double v);
int oracle_bf16_round(const double* in, int64_t n, double* out) {
    if (!in || !out || n < 0) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) out[i] = bf16_round(in[i]);
    return ORACLE_OK;
}

/* Threads the oracle's parallel loops use, and a way to set that count (the
 * results do not depend on it: every reduction runs in sample order). */
int oracle_num_threads(void) { return omp_get_max_threads(); }
int oracle_set_num_threads(int n) {
    if (n < 1) return ORACLE_EINVAL;
    omp_set_num_threads(n);
    return ORACLE_OK;
}

int64_t oracle_param_count(const oracle_net* net) {
    shapes_t sh;
    if (make_shapes(net, &sh) != ORACLE_OK) return -1;
    return sh.n_params;
}

/* Offset of layer l's weight (is_bias = 0) or bias (is_bias = 1); layers are
 * numbered conv1..convL, fc1, fc2. */
int64_t oracle_param_offset(const oracle_net* net, int32_t layer, int32_t is_bias) {
    shapes_t sh;
    if (make_shapes(net, &sh) != ORACLE_OK) return -1;
    if (layer < 0 || layer > net->n_conv + 1) return -1;
    return is_bias ? sh.b_off[layer] : sh.w_off[layer];
}

/* ------------------------------------------------------------------------ */
/* Layers for one sample.  Activations are [channel][y][x]. */

/* z[o][y][x] = b[o] + sum_{c,ky,kx} W[o][c][ky][kx] in[c][s*y+ky][s*x+kx] */
static void conv_forward(const double* in, int C, int H, int W_, const double* Wt,
                         const double* b, int O, int k, int s, int OH, int OW, double* z) {
    for (int o = 0; o < O; ++o)
        for (int y = 0; y < OH; ++y)
            for (int x = 0; x < OW; ++x) {
                double acc = b[o];
                for (int c = 0; c < C; ++c)
                    for (int ky = 0; ky < k; ++ky)
                        for (int kx = 0; kx < k; ++kx)
                            acc += Wt[((o * C + c) * k + ky) * k + kx] *
                                   in[(c * H + s * y + ky) * W_ + s * x + kx];
                z[(o * OH + y) * OW + x] = acc;
            }
}

/* Given dz = dL/dz, accumulate dL/dW and dL/db; if din is not NULL also
 * dL/d(in) (the transposed convolution: each output scatters W * dz back
 * onto the input window it read).  dzm is the dz that multiplies W and the
 * input (dz itself, or its bf16 rounding in the bf16-input variant); the
 * bias gradient sums dz. */
static void conv_backward(const double* in, int C, int H, int W_, const double* Wt,
                          int O, int k, int s, int OH, int OW, const double* dz, const double* dzm,
                          double* dW, double* db, double* din) {
    for (int o = 0; o < O; ++o)
        for (int y = 0; y < OH; ++y)
            for (int x = 0; x < OW; ++x) {
                double g = dzm[(o * OH + y) * OW + x];
                db[o] += dz[(o * OH + y) * OW + x];
                for (int c = 0; c < C; ++c)
                    for (int ky = 0; ky < k; ++ky)
                        for (int kx = 0; kx < k; ++kx) {
                            int64_t wi = ((o * C + c) * k + ky) * k + kx;
                            int64_t ii = (c * H + s * y + ky) * W_ + s * x + kx;
                            dW[wi] += g * in[ii];
                            if (din) din[ii] += g * Wt[wi];
                        }
            }
}

/* z[o] = b[o] + sum_i W[o][i] in[i] */
static void fc_forward(const double* in, int64_t n_in, const double* Wt, const double* b,
                       int n_out, double* z) {
    for (int o = 0; o < n_out; ++o) {
        double acc = b[o];
        for (int64_t i = 0; i < n_in; ++i) acc += Wt[(int64_t)o * n_in + i] * in[i];
        z[o] = acc;
    }
}

/* As conv_backward: dzm multiplies, dz feeds the bias gradient. */
static void fc_backward(const double* in, int64_t n_in, const double* Wt, int n_out,
                        const double* dz, const double* dzm, double* dW, double* db, double* din) {
    for (int o = 0; o < n_out; ++o) {
        db[o] += dz[o];
        for (int64_t i = 0; i < n_in; ++i) {
            dW[(int64_t)o * n_in + i] += dzm[o] * in[i];
            if (din) din[i] += dzm[o] * Wt[(int64_t)o * n_in + i];
        }
    }
}

static inline double relu(double v) { return v > 0.0 ? v : 0.0; }

/* v rounded to float32, then to bfloat16 (the upper 16 bits of a float32)
 * with round to nearest, ties to even; returned as double.  Non-finite
 * values are truncated (they do not occur here). */
static double bf16_round(double v) {
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7f800000u) != 0x7f800000u) u += 0x7fffu + ((u >> 16) & 1u);
    u &= 0xffff0000u;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* dst = the contraction operand of src: src itself, or its bf16 rounding. */
static const double* operand(const double* src, int64_t n, int bf16, double* dst) {
    if (!bf16) return src;
    for (int64_t i = 0; i < n; ++i) dst[i] = bf16_round(src[i]);
    return dst;
}

/* Per-sample activations: act[0] = scaled input, act[l+1] = ReLU output of
 * conv l, then fc1's pre-activation z and post-ReLU h, then Q. */
typedef struct {
    double* act[ORACLE_MAX_CONV + 1];
    double* zc[ORACLE_MAX_CONV];
    double* z1;
    double* h1;
    double* q;
    double* opnd[ORACLE_MAX_CONV + 1];  /* contraction operand of act[l] */
} acts_t;

static int acts_alloc(const oracle_net* net, const shapes_t* sh, acts_t* a) {
    memset(a, 0, sizeof(*a));
    for (int l = 0; l <= net->n_conv; ++l) {
        a->act[l] = (double*)calloc((size_t)sh->c[l] * sh->h[l] * sh->w[l], sizeof(double));
        a->opnd[l] = (double*)calloc((size_t)sh->c[l] * sh->h[l] * sh->w[l], sizeof(double));
        if (!a->act[l] || !a->opnd[l]) return ORACLE_ENOMEM;
        if (l < net->n_conv) {
            a->zc[l] = (double*)calloc((size_t)sh->c[l + 1] * sh->h[l + 1] * sh->w[l + 1], sizeof(double));
            if (!a->zc[l]) return ORACLE_ENOMEM;
        }
    }
    a->z1 = (double*)calloc(net->fc_hidden, sizeof(double));
    a->h1 = (double*)calloc(net->fc_hidden, sizeof(double));
    a->q = (double*)calloc(net->n_actions, sizeof(double));
    return (a->z1 && a->h1 && a->q) ? ORACLE_OK : ORACLE_ENOMEM;
}

static void acts_free(const oracle_net* net, acts_t* a) {
    for (int l = 0; l <= net->n_conv; ++l) {
        free(a->act[l]);
        free(a->opnd[l]);
        if (l < net->n_conv) free(a->zc[l]);
    }
    free(a->z1); free(a->h1); free(a->q);
}

/* Q(phi; theta) for one state of bytes; input x = byte / 255.  thw holds the
 * contraction operands of the conv and fc1 weights (theta itself, or its
 * bf16 rounding); biases and fc2 come from th.  a->opnd[l] receives the
 * operand of each layer input (the bytes are exact in bf16; x = byte/255
 * then equals the scale applied after the sum). */
static void forward_one(const oracle_net* net, const shapes_t* sh, const double* th,
                        const double* thw, const uint8_t* state, acts_t* a) {
    const int bf = net->bf16_inputs;
    int64_t n_in = (int64_t)sh->c[0] * sh->h[0] * sh->w[0];
    for (int64_t i = 0; i < n_in; ++i) a->act[0][i] = a->opnd[0][i] = (double)state[i] / 255.0;
    for (int l = 0; l < net->n_conv; ++l) {
        const double* x = l == 0 ? a->opnd[0]
                                 : operand(a->act[l], (int64_t)sh->c[l] * sh->h[l] * sh->w[l], bf, a->opnd[l]);
        conv_forward(x, sh->c[l], sh->h[l], sh->w[l], thw + sh->w_off[l], th + sh->b_off[l],
                     sh->c[l + 1], net->conv_k[l], net->conv_stride[l], sh->h[l + 1], sh->w[l + 1], a->zc[l]);
        int64_t n = (int64_t)sh->c[l + 1] * sh->h[l + 1] * sh->w[l + 1];
        for (int64_t i = 0; i < n; ++i) a->act[l + 1][i] = relu(a->zc[l][i]);
    }
    int L = net->n_conv;
    const double* x = operand(a->act[L], sh->flat, bf, a->opnd[L]);
    fc_forward(x, sh->flat, thw + sh->w_off[L], th + sh->b_off[L], net->fc_hidden, a->z1);
    for (int h = 0; h < net->fc_hidden; ++h) a->h1[h] = relu(a->z1[h]);
    fc_forward(a->h1, net->fc_hidden, th + sh->w_off[L + 1], th + sh->b_off[L + 1], net->n_actions, a->q);
}

/* The contraction operands of theta's conv and fc1 weights: theta itself, or
 * a new array with those weights rounded to bf16 (the caller frees it when
 * it differs from theta).  NULL when out of memory. */
static const double* weight_operands(const oracle_net* net, const shapes_t* sh, const double* th) {
    if (!net->bf16_inputs) return th;
    double* r = (double*)malloc(sizeof(double) * (size_t)sh->n_params);
    if (!r) return NULL;
    memcpy(r, th, sizeof(double) * (size_t)sh->n_params);
    for (int l = 0; l <= net->n_conv; ++l) {
        int64_t n = sh->b_off[l] - sh->w_off[l];
        for (int64_t i = 0; i < n; ++i) r[sh->w_off[l] + i] = bf16_round(th[sh->w_off[l] + i]);
    }
    return r;
}

/* ------------------------------------------------------------------------ */
/* How close each sample's forward pass comes to a ReLU kink.  For every ReLU
 * unit u (conv layers and the hidden fc layer) with pre-activation
 * z_u = b_u + sum_k w_uk x_k, the normalized margin is
 * |z_u| / (|b_u| + sum_k |w_uk x_k|): the distance to the kink in units of
 * the magnitude of the terms summed, which is the scale of any rounding
 * error in z_u.  Where it is below the working precision the ReLU derivative
 * is not decided by the arithmetic, and two correct implementations may
 * differ there.  Used by the tests to tell unique gradients from
 * precision-ambiguous ones. */

static double margin_of(double z, double den) {
    return den > 0.0 ? fabs(z) / den : (z == 0.0 ? 0.0 : INFINITY);
}

static void margin_one(const oracle_net* net, const shapes_t* sh, const double* th,
                       const uint8_t* state, acts_t* a, double* out) {
    double m = INFINITY;
    int64_t n_in = (int64_t)sh->c[0] * sh->h[0] * sh->w[0];
    for (int64_t i = 0; i < n_in; ++i) a->act[0][i] = (double)state[i] / 255.0;
    for (int l = 0; l < net->n_conv; ++l) {
        const double* W = th + sh->w_off[l];
        const double* b = th + sh->b_off[l];
        const int C = sh->c[l], H = sh->h[l], Wd = sh->w[l], O = sh->c[l + 1];
        const int k = net->conv_k[l], s = net->conv_stride[l], OH = sh->h[l + 1], OW = sh->w[l + 1];
        for (int o = 0; o < O; ++o)
            for (int y = 0; y < OH; ++y)
                for (int x = 0; x < OW; ++x) {
                    double z = b[o], den = fabs(b[o]);
                    for (int c = 0; c < C; ++c)
                        for (int ky = 0; ky < k; ++ky)
                            for (int kx = 0; kx < k; ++kx) {
                                double t = W[((o * C + c) * k + ky) * k + kx] *
                                           a->act[l][(c * H + s * y + ky) * Wd + s * x + kx];
                                z += t;
                                den += fabs(t);
                            }
                    double mu = margin_of(z, den);
                    if (mu < m) m = mu;
                    a->act[l + 1][(o * OH + y) * OW + x] = relu(z);
                }
    }
    int L = net->n_conv;
    const double* W1 = th + sh->w_off[L];
    const double* b1 = th + sh->b_off[L];
    for (int h = 0; h < net->fc_hidden; ++h) {
        double z = b1[h], den = fabs(b1[h]);
        for (int64_t i = 0; i < sh->flat; ++i) {
            double t = W1[(int64_t)h * sh->flat + i] * a->act[L][i];
            z += t;
            den += fabs(t);
        }
        double mu = margin_of(z, den);
        if (mu < m) m = mu;
    }
    *out = m;
}

/* margin_out[j] = smallest normalized ReLU margin of Q(states[j]; theta). */
int oracle_relu_margins(const oracle_net* net, const double* theta, const uint8_t* states,
                        int64_t batch, double* margin_out) {
    shapes_t sh;
    if (make_shapes(net, &sh) != ORACLE_OK || !theta || !states || !margin_out || batch < 0)
        return ORACLE_EINVAL;
    int64_t in_bytes = (int64_t)sh.c[0] * sh.h[0] * sh.w[0];
    int err = ORACLE_OK;
    #pragma omp parallel
    {
        acts_t a;
        int e = acts_alloc(net, &sh, &a);
        if (e != ORACLE_OK) {
            #pragma omp atomic write
            err = e;
        } else {
            #pragma omp for schedule(static)
            for (int64_t j = 0; j < batch; ++j)
                margin_one(net, &sh, theta, states + j * in_bytes, &a, margin_out + j);
        }
        acts_free(net, &a);
    }
    return err;
}

/* ------------------------------------------------------------------------ */

/* Minibatch gather from a replay memory (Sec. III.C, Alg. 1).  Record i
 * starts at frames + i * record_stride and holds rec_bytes bytes (the
 * stacked frames phi_i).  Transition i is (phi_i, a_i, r_i, term_i,
 * phi_{i+1}), so valid indices are 0 .. size-2; term_i = 1 marks phi_{i+1}
 * as terminal.  s_next may be NULL (states only). */
int oracle_replay_gather(const uint8_t* frames, int64_t record_stride, int64_t rec_bytes,
                         int64_t size, const uint8_t* action, const int8_t* reward,
                         const uint8_t* terminal, const int64_t* idx, int64_t batch,
                         int64_t max_index, uint8_t* s, uint8_t* s_next, int32_t* a, float* r,
                         uint8_t* t) {
    if (!frames || !idx || batch < 0 || rec_bytes <= 0) return ORACLE_EINVAL;
    for (int64_t j = 0; j < batch; ++j) {
        int64_t i = idx[j];
        if (i < 0 || i > max_index || i >= size) return ORACLE_ERANGE;
        memcpy(s + j * rec_bytes, frames + i * record_stride, (size_t)rec_bytes);
        if (s_next) memcpy(s_next + j * rec_bytes, frames + (i + 1) * record_stride, (size_t)rec_bytes);
        if (a) a[j] = action[i];
        if (r) r[j] = (float)reward[i];
        if (t) t[j] = terminal[i];
    }
    return ORACLE_OK;
}

/* Q values, q_out[B][A]. */
int oracle_forward_q(const oracle_net* net, const double* theta, const uint8_t* states,
                     int64_t batch, double* q_out) {
    shapes_t sh;
    if (make_shapes(net, &sh) != ORACLE_OK || !theta || !states || !q_out || batch < 0)
        return ORACLE_EINVAL;
    int64_t in_bytes = (int64_t)sh.c[0] * sh.h[0] * sh.w[0];
    const double* thw = weight_operands(net, &sh, theta);
    if (!thw) return ORACLE_ENOMEM;
    int err = ORACLE_OK;
    #pragma omp parallel
    {
        acts_t a;
        int e = acts_alloc(net, &sh, &a);
        if (e != ORACLE_OK) {
            #pragma omp atomic write
            err = e;
        } else {
            #pragma omp for schedule(static)
            for (int64_t j = 0; j < batch; ++j) {
                forward_one(net, &sh, theta, thw, states + j * in_bytes, &a);
                for (int k = 0; k < net->n_actions; ++k) q_out[j * net->n_actions + k] = a.q[k];
            }
        }
        acts_free(net, &a);
    }
    if (thw != theta) free((void*)thw);
    return err;
}

/* Epsilon-greedy action choice (Sec. III.B, Alg. 1).  Reading of the paper:
 * "max_a Q" in the action rule means argmax; ties go to the lowest action
 * index; the random action is uniform over all A actions.  With draw
 * w = draws[j] (64 uniform bits supplied by the caller): explore iff
 * (w >> 32) < floor(epsilon * 2^32); the random action is
 * ((w & 0xffffffff) * A) >> 32.  draws may be NULL when epsilon == 0. */
int oracle_select_actions(const double* q, int64_t batch, int32_t n_actions, double epsilon,
                          const uint64_t* draws, int32_t* actions) {
    if (!q || !actions || n_actions <= 0 || batch < 0) return ORACLE_EINVAL;
    if (!(epsilon >= 0.0 && epsilon <= 1.0)) return ORACLE_EINVAL;
    double te = floor(epsilon * 4294967296.0);
    uint64_t thresh = te >= 4294967296.0 ? 4294967296ull : (uint64_t)te;
    if (thresh > 0 && !draws) return ORACLE_EINVAL;
    for (int64_t j = 0; j < batch; ++j) {
        const double* qj = q + j * n_actions;
        int best = 0;
        for (int k = 1; k < n_actions; ++k)
            if (qj[k] > qj[best]) best = k;
        if (thresh > 0 && (draws[j] >> 32) < thresh)
            best = (int)(((draws[j] & 0xffffffffull) * (uint64_t)n_actions) >> 32);
        actions[j] = best;
    }
    return ORACLE_OK;
}

/* The worker's minibatch gradient (Alg. 1):
 *   y_j = r_j                                   if term_j,
 *   y_j = r_j + gamma * max_a' Q(s'_j, a'; theta_tgt)  otherwise;
 *   loss = (1/B) sum_j 1/2 (Q(s_j, a_j; theta) - y_j)^2;
 *   grad = d loss / d theta with y_j held constant.
 * Readings: the loss and gradient carry the 1/2 and 1/b of Alg. 1 rather
 * than the bare expectation of Eq. (1); the target network theta_tgt is the
 * held copy of the parameters (theta-hat), never differentiated, even when
 * it equals theta; ReLU'(0) = 0.
 * Outputs: grad [p] (overwritten), loss [1], and optional q_all [B][A]
 * (Q(s_j, .; theta)), qn_all [B][A] (Q(s'_j, .; theta_tgt)), y [B]. */
int oracle_td_gradient(const oracle_net* net, const double* theta, const double* theta_tgt,
                       const uint8_t* s, const uint8_t* s_next, const int32_t* action,
                       const float* reward, const uint8_t* terminal, int64_t batch, double gamma,
                       double* grad, double* loss, double* q_all, double* qn_all, double* y_out) {
    shapes_t sh;
    if (make_shapes(net, &sh) != ORACLE_OK || !theta || !theta_tgt || !s || !s_next || !action ||
        !reward || !terminal || !grad || !loss || batch <= 0)
        return ORACLE_EINVAL;
    for (int64_t j = 0; j < batch; ++j)
        if (action[j] < 0 || action[j] >= net->n_actions) return ORACLE_ERANGE;
    const int64_t P = sh.n_params;
    const int64_t in_bytes = (int64_t)sh.c[0] * sh.h[0] * sh.w[0];
    const int L = net->n_conv, H = net->fc_hidden, A = net->n_actions;
    int nthreads = omp_get_max_threads();
    if (nthreads > batch) nthreads = (int)batch;
    /* Per-sample gradients are computed in parallel, nthreads at a time, and
     * added to the total strictly in sample order. */
    const int bf = net->bf16_inputs;
    double* g = (double*)calloc((size_t)nthreads * (size_t)P, sizeof(double));
    double* lj = (double*)calloc((size_t)batch, sizeof(double));
    const double* thw = weight_operands(net, &sh, theta);
    const double* ttw = weight_operands(net, &sh, theta_tgt);
    if (!g || !lj || !thw || !ttw) {
        free(g); free(lj);
        if (thw && thw != theta) free((void*)thw);
        if (ttw && ttw != theta_tgt) free((void*)ttw);
        return ORACLE_ENOMEM;
    }
    memset(grad, 0, sizeof(double) * (size_t)P);
    int err = ORACLE_OK;
    for (int64_t j0 = 0; j0 < batch && err == ORACLE_OK; j0 += nthreads) {
        int64_t jn = batch - j0 < nthreads ? batch - j0 : nthreads;
        #pragma omp parallel num_threads(nthreads)
        {
            acts_t a, an;
            int e1 = acts_alloc(net, &sh, &a), e2 = acts_alloc(net, &sh, &an);
            double *d_cur = (double*)calloc((size_t)sh.max_act, sizeof(double));
            double *d_prev = (double*)calloc((size_t)sh.max_act, sizeof(double));
            double *d_opnd = (double*)calloc((size_t)sh.max_act, sizeof(double));
            double *dq = (double*)calloc((size_t)A, sizeof(double));
            double *dh = (double*)calloc((size_t)H, sizeof(double));
            if (e1 || e2 || !d_cur || !d_prev || !d_opnd || !dq || !dh) {
                #pragma omp atomic write
                err = ORACLE_ENOMEM;
            } else {
                #pragma omp for schedule(static)
                for (int64_t t = 0; t < jn; ++t) {
                    int64_t j = j0 + t;
                    double* gj = g + (size_t)t * (size_t)P;
                    memset(gj, 0, sizeof(double) * (size_t)P);
                    /* target from the held network on the next state */
                    forward_one(net, &sh, theta_tgt, ttw, s_next + j * in_bytes, &an);
                    double m = an.q[0];
                    for (int k = 1; k < A; ++k) if (an.q[k] > m) m = an.q[k];
                    double y = terminal[j] ? (double)reward[j] : (double)reward[j] + gamma * m;
                    /* prediction from the learned network on the state */
                    forward_one(net, &sh, theta, thw, s + j * in_bytes, &a);
                    double diff = a.q[action[j]] - y;
                    lj[j] = 0.5 * diff * diff / (double)batch;
                    if (q_all) for (int k = 0; k < A; ++k) q_all[j * A + k] = a.q[k];
                    if (qn_all) for (int k = 0; k < A; ++k) qn_all[j * A + k] = an.q[k];
                    if (y_out) y_out[j] = y;
                    /* dL/dQ_j: nonzero only at the taken action */
                    for (int k = 0; k < A; ++k) dq[k] = (k == action[j]) ? diff / (double)batch : 0.0;
                    /* fc2 (linear) */
                    memset(dh, 0, sizeof(double) * (size_t)H);
                    fc_backward(a.h1, H, theta + sh.w_off[L + 1], A, dq, dq, gj + sh.w_off[L + 1],
                                gj + sh.b_off[L + 1], dh);
                    for (int h = 0; h < H; ++h) dh[h] = a.z1[h] > 0.0 ? dh[h] : 0.0;
                    /* fc1: products with the contraction operands of dh, its
                     * input and its weights */
                    memset(d_cur, 0, sizeof(double) * (size_t)sh.flat);
                    fc_backward(bf ? a.opnd[L] : a.act[L], sh.flat,
                                thw + sh.w_off[L], H, dh, operand(dh, H, bf, d_opnd), gj + sh.w_off[L],
                                gj + sh.b_off[L], d_cur);
                    /* conv layers, last to first; no gradient into the input */
                    for (int l = L - 1; l >= 0; --l) {
                        int64_t n_out = (int64_t)sh.c[l + 1] * sh.h[l + 1] * sh.w[l + 1];
                        for (int64_t i = 0; i < n_out; ++i) d_cur[i] = a.zc[l][i] > 0.0 ? d_cur[i] : 0.0;
                        int64_t n_in = (int64_t)sh.c[l] * sh.h[l] * sh.w[l];
                        if (l > 0) memset(d_prev, 0, sizeof(double) * (size_t)n_in);
                        conv_backward(bf ? a.opnd[l] : a.act[l], sh.c[l], sh.h[l], sh.w[l], thw + sh.w_off[l],
                                      sh.c[l + 1], net->conv_k[l], net->conv_stride[l], sh.h[l + 1],
                                      sh.w[l + 1], d_cur, operand(d_cur, n_out, bf, d_opnd),
                                      gj + sh.w_off[l], gj + sh.b_off[l], l > 0 ? d_prev : NULL);
                        double* tmp = d_cur; d_cur = d_prev; d_prev = tmp;
                    }
                }
            }
            acts_free(net, &a); acts_free(net, &an);
            free(d_cur); free(d_prev); free(d_opnd); free(dq); free(dh);
        }
        for (int64_t t = 0; t < jn && err == ORACLE_OK; ++t) {
            const double* gj = g + (size_t)t * (size_t)P;
            for (int64_t i = 0; i < P; ++i) grad[i] += gj[i];
        }
    }
    double ls = 0.0;
    for (int64_t j = 0; j < batch; ++j) ls += lj[j];
    *loss = ls;
    free(g); free(lj);
    if (thw != theta) free((void*)thw);
    if (ttw != theta_tgt) free((void*)ttw);
    return err;
}

/* Parameter-server update, elementwise, computed in double from the float32
 * stored state; theta_out and state are rounded to float32 on store.
 *   RULE_SGD:     theta <- theta - lr g  (the garbled descent rule of
 *                 Sec. III.B read as a step against the gradient).
 *   RULE_RMSPROP: Alg. 2: r <- decay r + (1 - decay) g^2 (decay 0.9 in the
 *                 paper), then theta <- theta - lr g / sqrt(r) using the new
 *                 r.  Alg. 2 has no epsilon; where the new r is exactly 0
 *                 (every gradient so far was 0) the parameter is unchanged.
 *   RULE_ADAGRAD: G <- G + g^2; theta <- theta - lr g / (sqrt(G) + eps)
 *                 (AdaGrad is only named in Sec. IV.D.2; eps sits outside
 *                 the square root).
 * state may be NULL for SGD.  theta_out may equal theta_in. */
int oracle_apply_update(int32_t rule, const float* theta_in, float* theta_out, float* state,
                        const double* grad, int64_t n, double lr, double decay, double eps) {
    if (!theta_in || !theta_out || !grad || n < 0) return ORACLE_EINVAL;
    if (rule != RULE_SGD && !state) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        double th = (double)theta_in[i], g = grad[i];
        if (rule == RULE_SGD) {
            th = th - lr * g;
        } else if (rule == RULE_RMSPROP) {
            double r = decay * (double)state[i] + (1.0 - decay) * g * g;
            state[i] = (float)r;
            if (r > 0.0) th = th - lr * g / sqrt(r);
        } else if (rule == RULE_ADAGRAD) {
            double G = (double)state[i] + g * g;
            state[i] = (float)G;
            th = th - lr * g / (sqrt(G) + eps);
        } else {
            return ORACLE_EINVAL;
        }
        theta_out[i] = (float)th;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* The actor side of Alg. 1 ("Execute action a_t and observe reward r_t and
 * frame x_{t+1}; store the experience in D").  The game is Snake as Sec. V.A
 * describes it: an n x n array; the snake starts with a body of length two
 * and grows by one when it eats an apple, which scores +1; hitting itself
 * ends the game and scores -1.  Readings where the text is silent:
 *  - the board wraps around at its edges (a torus), so hitting itself is the
 *    only way a game ends, as the text says;
 *  - actions 0..3 set the heading (up, right, down, left); any other action,
 *    and the reverse of the current heading, keep it;
 *  - the tail leaves its cell in the same move, so moving into it is not a
 *    collision; when the snake eats, the tail stays;
 *  - random placement uses two caller-supplied 64-bit words per game and
 *    step: a new game puts the head on cell floor(lo32(w0) * n^2 / 2^32)
 *    with heading hi2(w0), the second body cell behind it; an apple goes to
 *    the k-th free cell in row-major order, k = floor(hi32(w1) * free / 2^32);
 *  - a finished game restarts at once; the experience that ended it stores
 *    the new game's first state as its next state (its target is r alone, so
 *    that state is never evaluated);
 *  - a frame is 84 x 84 bytes, each cell a 7 x 7 block: 0 empty, 128 body,
 *    255 head, 192 apple; a state stacks the last four frames, oldest first,
 *    and a new game's state is four copies of its first frame. */

#define SNAKE_N 12
#define SNAKE_CELLS (SNAKE_N * SNAKE_N)
#define SNAKE_PX 7
#define SNAKE_FRAME (84 * 84)

typedef struct {
    int32_t body[SNAKE_CELLS]; /* cell indices, body[0] the head */
    int32_t len, heading, apple;
} oracle_snake;

static const int snake_dy[4] = {-1, 0, 1, 0};
static const int snake_dx[4] = {0, 1, 0, -1};

static int snake_move(int cell, int heading) {
    int y = cell / SNAKE_N, x = cell % SNAKE_N;
    y = (y + snake_dy[heading] + SNAKE_N) % SNAKE_N;
    x = (x + snake_dx[heading] + SNAKE_N) % SNAKE_N;
    return y * SNAKE_N + x;
}

static int snake_on_body(const oracle_snake* g, int cell, int upto) {
    for (int i = 0; i < upto; ++i)
        if (g->body[i] == cell) return 1;
    return 0;
}

static void snake_place_apple(oracle_snake* g, uint64_t w1) {
    int free_cells = SNAKE_CELLS - g->len;
    uint64_t k = ((w1 >> 32) * (uint64_t)free_cells) >> 32;
    for (int c = 0; c < SNAKE_CELLS; ++c) {
        if (snake_on_body(g, c, g->len)) continue;
        if (k == 0) { g->apple = c; return; }
        --k;
    }
    g->apple = -1; /* the board is full */
}

static void snake_new_game(oracle_snake* g, uint64_t w0, uint64_t w1) {
    int head = (int)(((w0 & 0xffffffffull) * (uint64_t)SNAKE_CELLS) >> 32);
    g->heading = (int)(w0 >> 62);
    g->body[0] = head;
    g->body[1] = snake_move(head, (g->heading + 2) % 4);
    g->len = 2;
    snake_place_apple(g, w1);
}

static void snake_render(const oracle_snake* g, uint8_t* frame) {
    for (int p = 0; p < SNAKE_FRAME; ++p) {
        int y = p / 84, x = p % 84;
        int cell = (y / SNAKE_PX) * SNAKE_N + x / SNAKE_PX;
        uint8_t v = 0;
        if (cell == g->apple) v = 192;
        if (snake_on_body(g, cell, g->len)) v = 128;
        if (cell == g->body[0]) v = 255;
        frame[p] = v;
    }
}

/* New games for every env: states [E][4][84][84] get four copies of the
 * first frame.  draws: [E][2]. */
int oracle_snake_reset(oracle_snake* games, int64_t E, const uint64_t* draws, uint8_t* states) {
    if (!games || !draws || !states || E < 0) return ORACLE_EINVAL;
    for (int64_t e = 0; e < E; ++e) {
        snake_new_game(&games[e], draws[2 * e], draws[2 * e + 1]);
        uint8_t* st = states + e * 4 * SNAKE_FRAME;
        snake_render(&games[e], st);
        for (int f = 1; f < 4; ++f) memcpy(st + f * SNAKE_FRAME, st, SNAKE_FRAME);
    }
    return ORACLE_OK;
}

/* One step of every game with its action; states advance by one frame (or
 * restart on a finished game).  reward [E] (float), terminal [E]. */
int oracle_snake_step(oracle_snake* games, int64_t E, const int32_t* actions, const uint64_t* draws,
                      uint8_t* states, float* reward, uint8_t* terminal) {
    if (!games || !actions || !draws || !states || !reward || !terminal || E < 0) return ORACLE_EINVAL;
    for (int64_t e = 0; e < E; ++e) {
        oracle_snake* g = &games[e];
        int a = actions[e];
        if (a >= 0 && a < 4 && a != (g->heading + 2) % 4) g->heading = a;
        int nh = snake_move(g->body[0], g->heading);
        float r = 0.f;
        uint8_t term = 0;
        int eats = nh == g->apple;
        /* every segment but the tail, which moves away unless the snake eats */
        if (snake_on_body(g, nh, eats ? g->len : g->len - 1)) {
            r = -1.f;
            term = 1;
        } else {
            int keep = eats ? g->len : g->len - 1;
            for (int i = keep; i > 0; --i) g->body[i] = g->body[i - 1];
            g->body[0] = nh;
            if (eats) {
                g->len += 1;
                r = 1.f;
                snake_place_apple(g, draws[2 * e + 1]);
            }
        }
        uint8_t* st = states + e * 4 * SNAKE_FRAME;
        if (term) {
            snake_new_game(g, draws[2 * e], draws[2 * e + 1]);
            snake_render(g, st);
            for (int f = 1; f < 4; ++f) memcpy(st + f * SNAKE_FRAME, st, SNAKE_FRAME);
        } else {
            memmove(st, st + SNAKE_FRAME, 3 * SNAKE_FRAME);
            snake_render(g, st + 3 * SNAKE_FRAME);
        }
        reward[e] = r;
        terminal[e] = term;
    }
    return ORACLE_OK;
}

/* The replay memory keeps the last N states of each game (Sec. III.C): game
 * e owns records e*(N+1) .. e*(N+1)+N of `frames` (rec_bytes each); state t
 * of the game lives in slot t mod N, and slot N repeats slot 0, so the
 * successor of every slot is the next record.  Experience t of game e is
 * (state t, a_t, r_t, term_t, state t+1): its side fields are stored at the
 * record of state t.  t = -1 stores the initial states only. */
int oracle_replay_append(uint8_t* frames, int64_t rec_bytes, int64_t E, int64_t N, int64_t t,
                         const uint8_t* states, const int32_t* actions, const float* reward,
                         const uint8_t* terminal, uint8_t* action_mem, int8_t* reward_mem,
                         uint8_t* terminal_mem) {
    if (!frames || !states || E < 0 || N < 2 || t < -1 || rec_bytes <= 0) return ORACLE_EINVAL;
    for (int64_t e = 0; e < E; ++e) {
        int64_t base = e * (N + 1);
        int64_t slot = (t + 1) % N;
        memcpy(frames + (base + slot) * rec_bytes, states + e * rec_bytes, (size_t)rec_bytes);
        if (slot == 0) memcpy(frames + (base + N) * rec_bytes, states + e * rec_bytes, (size_t)rec_bytes);
        if (t >= 0) {
            int64_t r = base + t % N;
            action_mem[r] = (uint8_t)actions[e];
            reward_mem[r] = (int8_t)reward[e];
            terminal_mem[r] = terminal[e];
        }
    }
    return ORACLE_OK;
}

/* Exploration rate of Alg. 1 at iteration n: q = max((N_max - n)/N_max, 0),
 * epsilon = (1 - q) eps_min + q eps_max. */
double oracle_anneal_epsilon(int64_t n, int64_t n_max, double eps_min, double eps_max) {
    double q = n_max > 0 ? (double)(n_max - n) / (double)n_max : 0.0;
    if (q < 0.0) q = 0.0;
    return (1.0 - q) * eps_min + q * eps_max;
}

/* ------------------------------------------------------------------------ */
/* Preprocessing phi (Sec. III.A): raw RGB frames are gray-scaled and
 * down-sampled to 84 x 84.  The text names the steps only; the reading:
 * gray = (299 R + 587 G + 114 B + 500) / 1000 in integers (ITU-R BT.601
 * weights, rounded half up), then the 84f x 84f window at (top, left) is
 * averaged over f x f blocks, (sum + f*f/2) / (f*f), rounded half up.
 * rgb: uint8 [n][h][w][3]; out: uint8 [n][84][84]. */
int oracle_preprocess(const uint8_t* rgb, int64_t n, int32_t h, int32_t w, int32_t top, int32_t left,
                      int32_t f, uint8_t* out) {
    if (!rgb || !out || n < 0 || f < 1 || top < 0 || left < 0 || top + 84 * f > h || left + 84 * f > w)
        return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        const uint8_t* fr = rgb + i * (int64_t)h * w * 3;
        for (int y = 0; y < 84; ++y)
            for (int x = 0; x < 84; ++x) {
                int64_t sum = 0;
                for (int dy = 0; dy < f; ++dy)
                    for (int dx = 0; dx < f; ++dx) {
                        const uint8_t* px = fr + ((int64_t)(top + y * f + dy) * w + (left + x * f + dx)) * 3;
                        sum += (299 * px[0] + 587 * px[1] + 114 * px[2] + 500) / 1000;
                    }
                out[(i * 84 + y) * 84 + x] = (uint8_t)((sum + (f * f) / 2) / (f * f));
            }
    }
    return ORACLE_OK;
}
