/* CPython-level calls of whtmix_forward_ex and whtmix_forward_separable.
 *
 * Argument marshalling only: Python integers become the C ABI's pointers,
 * sizes and codes, and the library's status comes back as an int.  The
 * functions are reached through addresses that the Python binding takes
 * from the libwhtmix.so it has already loaded (bind()), so there is one
 * instance of the library and of its per-stream workspaces.  A ctypes call
 * of these entry points costs about 1.2 us of Python overhead; this one about
 * 0.15 us, which matters for slices whose whole call takes a few
 * microseconds.  Host code only (no HIP); the GIL is released around the
 * call as ctypes does. */
#define PY_SSIZE_T_CLEAN
#include <Python.h>
#include <stdint.h>

typedef int (*forward_ex_fn)(const void *x, const float *gain, void *y, int64_t B, int64_t N,
                             int64_t C, int dtype, void *stream, const void *options);
typedef int (*forward_sep_fn)(const void *x, const float *gt, const float *gc, void *y,
                              int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                              const void *options);

static forward_ex_fn g_forward_ex;
static forward_sep_fn g_forward_sep;

/* A pointer argument: an int (an address) or None (NULL). */
static int as_ptr(PyObject *o, void **out)
{
    if (o == Py_None) {
        *out = NULL;
        return 0;
    }
    if (!PyLong_Check(o)) {
        PyErr_SetString(PyExc_TypeError, "pointer arguments must be int or None");
        return -1;
    }
    *out = PyLong_AsVoidPtr(o);
    return PyErr_Occurred() ? -1 : 0;
}

static int as_i64(PyObject *o, int64_t *out)
{
    const long long v = PyLong_AsLongLong(o);
    if (v == -1 && PyErr_Occurred())
        return -1;
    *out = (int64_t)v;
    return 0;
}

static int as_int(PyObject *o, int *out)
{
    const long v = PyLong_AsLong(o);
    if (v == -1 && PyErr_Occurred())
        return -1;
    if (v < INT32_MIN || v > INT32_MAX) {
        PyErr_SetString(PyExc_OverflowError, "int argument out of range");
        return -1;
    }
    *out = (int)v;
    return 0;
}

/* bind(forward_ex_address, forward_separable_address) */
static PyObject *bind(PyObject *self, PyObject *const *args, Py_ssize_t nargs)
{
    (void)self;
    void *f = NULL, *s = NULL;
    if (nargs != 2) {
        PyErr_SetString(PyExc_TypeError, "bind() takes 2 addresses");
        return NULL;
    }
    if (as_ptr(args[0], &f) || as_ptr(args[1], &s))
        return NULL;
    if (!f || !s) {
        PyErr_SetString(PyExc_ValueError, "bind() needs non-null addresses");
        return NULL;
    }
    g_forward_ex = (forward_ex_fn)f;
    g_forward_sep = (forward_sep_fn)s;
    Py_RETURN_NONE;
}

/* forward_ex(x, gain, y, B, N, C, dtype, stream, options) -> status */
static PyObject *forward_ex(PyObject *self, PyObject *const *args, Py_ssize_t nargs)
{
    (void)self;
    void *x, *g, *y, *st, *opt;
    int64_t B, N, C;
    int dt, status;
    if (nargs != 9) {
        PyErr_SetString(PyExc_TypeError, "forward_ex() takes 9 arguments");
        return NULL;
    }
    if (!g_forward_ex) {
        PyErr_SetString(PyExc_RuntimeError, "forward_ex() called before bind()");
        return NULL;
    }
    if (as_ptr(args[0], &x) || as_ptr(args[1], &g) || as_ptr(args[2], &y) ||
        as_i64(args[3], &B) || as_i64(args[4], &N) || as_i64(args[5], &C) ||
        as_int(args[6], &dt) || as_ptr(args[7], &st) || as_ptr(args[8], &opt))
        return NULL;
    Py_BEGIN_ALLOW_THREADS
    status = g_forward_ex(x, (const float *)g, y, B, N, C, dt, st, opt);
    Py_END_ALLOW_THREADS
    return PyLong_FromLong(status);
}

/* forward_separable(x, gain_t, gain_c, y, B, N, C, dtype, stream, options) -> status */
static PyObject *forward_separable(PyObject *self, PyObject *const *args, Py_ssize_t nargs)
{
    (void)self;
    void *x, *gt, *gc, *y, *st, *opt;
    int64_t B, N, C;
    int dt, status;
    if (nargs != 10) {
        PyErr_SetString(PyExc_TypeError, "forward_separable() takes 10 arguments");
        return NULL;
    }
    if (!g_forward_sep) {
        PyErr_SetString(PyExc_RuntimeError, "forward_separable() called before bind()");
        return NULL;
    }
    if (as_ptr(args[0], &x) || as_ptr(args[1], &gt) || as_ptr(args[2], &gc) ||
        as_ptr(args[3], &y) || as_i64(args[4], &B) || as_i64(args[5], &N) ||
        as_i64(args[6], &C) || as_int(args[7], &dt) || as_ptr(args[8], &st) ||
        as_ptr(args[9], &opt))
        return NULL;
    Py_BEGIN_ALLOW_THREADS
    status = g_forward_sep(x, (const float *)gt, (const float *)gc, y, B, N, C, dt, st, opt);
    Py_END_ALLOW_THREADS
    return PyLong_FromLong(status);
}

static PyMethodDef methods[] = {
    {"bind", (PyCFunction)(void (*)(void))bind, METH_FASTCALL,
     "bind(forward_ex_address, forward_separable_address)"},
    {"forward_ex", (PyCFunction)(void (*)(void))forward_ex, METH_FASTCALL,
     "forward_ex(x, gain, y, B, N, C, dtype, stream, options) -> status"},
    {"forward_separable", (PyCFunction)(void (*)(void))forward_separable, METH_FASTCALL,
     "forward_separable(x, gain_t, gain_c, y, B, N, C, dtype, stream, options) -> status"},
    {NULL, NULL, 0, NULL}};

static struct PyModuleDef module = {PyModuleDef_HEAD_INIT, "_whtmix_call",
                                    "CPython-level calls of the WHTMix forward entry points",
                                    -1, methods, NULL, NULL, NULL, NULL};

PyMODINIT_FUNC PyInit__whtmix_call(void) { return PyModule_Create(&module); }
