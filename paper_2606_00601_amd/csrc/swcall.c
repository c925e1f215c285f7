/* swcall.c -- the Python binding's call path into libscanweaver.
 *
 * One METH_FASTCALL function per entry point of include/scanweaver.h, with
 * the entry point's name and arguments: pointers as Python ints (device
 * addresses) or None for NULL, sizes and enums as ints.  Each function only
 * converts its arguments and calls the entry point with the GIL released;
 * it returns the status (or the string / handle the entry point returns).
 * A ctypes call spends about a microsecond converting seven arguments; this
 * path spends tens of nanoseconds, which matters for launch-sized calls.
 */
#define PY_SSIZE_T_CLEAN
#include <Python.h>
#include <limits.h>
#include <string.h>

#include "scanweaver.h"

typedef union {
  void* p;
  long long l;
  int i;
} Arg;

/* Convert args[0..n) by fmt: 'P' pointer (int or None), 'L' int64, 'I' int. */
static int parse(PyObject* const* args, Py_ssize_t n, const char* fmt, Arg* out,
                 const char* name) {
  const Py_ssize_t k = (Py_ssize_t)strlen(fmt);
  if (n != k) {
    PyErr_Format(PyExc_TypeError, "%s takes %zd arguments (%zd given)", name, k, n);
    return 0;
  }
  for (Py_ssize_t i = 0; i < k; ++i) {
    PyObject* o = args[i];
    if (fmt[i] == 'P') {
      if (o == Py_None) {
        out[i].p = NULL;
        continue;
      }
      if (!PyLong_Check(o)) {
        PyErr_Format(PyExc_TypeError, "%s: argument %zd must be an address (int) or None",
                     name, i);
        return 0;
      }
      out[i].p = PyLong_AsVoidPtr(o);
      if (PyErr_Occurred()) return 0;
    } else {
      if (!PyLong_Check(o)) {
        PyErr_Format(PyExc_TypeError, "%s: argument %zd must be an int", name, i);
        return 0;
      }
      const long long v = PyLong_AsLongLong(o);
      if (v == -1 && PyErr_Occurred()) return 0;
      if (fmt[i] == 'I') {
        if (v < INT_MIN || v > INT_MAX) {
          PyErr_Format(PyExc_OverflowError, "%s: argument %zd does not fit an int", name, i);
          return 0;
        }
        out[i].i = (int)v;
      } else {
        out[i].l = v;
      }
    }
  }
  return 1;
}

/* The body of a wrapper: parse, call with the GIL released, return the status. */
#define SW_CALL(NAME, FMT, NARGS, CALL)                                 \
  static PyObject* py_##NAME(PyObject* self, PyObject* const* args,     \
                             Py_ssize_t nargs) {                        \
    (void)self;                                                         \
    Arg v[NARGS + 1];                                                   \
    if (!parse(args, nargs, FMT, v, #NAME)) return NULL;                \
    int st;                                                             \
    Py_BEGIN_ALLOW_THREADS st = CALL;                                   \
    Py_END_ALLOW_THREADS return PyLong_FromLong(st);                    \
  }

#define AP(k) v[k].p
#define AL(k) v[k].l
#define AI(k) v[k].i

SW_CALL(sw_affine_scan, "PPPPLLL", 7, sw_affine_scan(AP(0), AP(1), AP(2), AP(3), AL(4), AL(5), AL(6)))
SW_CALL(sw_affine_scan_i32, "PPPPLLL", 7,
        sw_affine_scan_i32(AP(0), AP(1), AP(2), AP(3), AL(4), AL(5), AL(6)))
SW_CALL(sw_affine_scan_noalloc, "PPPPLLL", 7,
        sw_affine_scan_noalloc(AP(0), AP(1), AP(2), AP(3), AL(4), AL(5), AL(6)))
SW_CALL(sw_affine_scan_schedule, "PPPPLLLI", 8,
        sw_affine_scan_schedule(AP(0), AP(1), AP(2), AP(3), AL(4), AL(5), AL(6), AI(7)))
SW_CALL(sw_affine_scan_schedule_i32, "PPPPLLLI", 8,
        sw_affine_scan_schedule_i32(AP(0), AP(1), AP(2), AP(3), AL(4), AL(5), AL(6), AI(7)))
SW_CALL(sw_affine_scan_proj, "PPPPPPPLLL", 10,
        sw_affine_scan_proj(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AL(7), AL(8), AL(9)))
SW_CALL(sw_affine_scan_proj_i32, "PPPPPPPLLL", 10,
        sw_affine_scan_proj_i32(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AL(7), AL(8), AL(9)))
SW_CALL(sw_selective_scan_fwd, "PPPPPPPPLLLL", 12,
        sw_selective_scan_fwd(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AL(8), AL(9),
                              AL(10), AL(11)))
SW_CALL(sw_selective_scan_fwd_bf16, "PPPPPPPPLLLL", 12,
        sw_selective_scan_fwd_bf16(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AL(8), AL(9),
                                   AL(10), AL(11)))
SW_CALL(sw_selective_scan_fwd_schedule, "PPPPPPPPLLLLII", 14,
        sw_selective_scan_fwd_schedule(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AL(8),
                                       AL(9), AL(10), AL(11), AI(12), AI(13)))
SW_CALL(sw_selective_scan_fwd_ex, "PPPPPPPPPPPLLLLIII", 18,
        sw_selective_scan_fwd_ex(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AP(8), AP(9),
                                 AP(10), AL(11), AL(12), AL(13), AL(14), AI(15), AI(16), AI(17)))
SW_CALL(sw_selective_scan_fwd_train, "PPPPPPPPPPPPPLLLLIII", 20,
        sw_selective_scan_fwd_train(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AP(8), AP(9),
                                    AP(10), AP(11), AP(12), AL(13), AL(14), AL(15), AL(16), AI(17),
                                    AI(18), AI(19)))
SW_CALL(sw_selective_scan_plan, "LLLLIIIIPPPP", 12,
        sw_selective_scan_plan(AL(0), AL(1), AL(2), AL(3), AI(4), AI(5), AI(6), AI(7), AP(8), AP(9),
                               AP(10), AP(11)))
SW_CALL(sw_selective_scan_bwd, "PPPPPPPPPPPPPPPPPPPPPPLLLLIII", 29,
        sw_selective_scan_bwd(AP(0), AP(1), AP(2), AP(3), AP(4), AP(5), AP(6), AP(7), AP(8), AP(9), AP(10),
                              AP(11), AP(12), AP(13), AP(14), AP(15), AP(16), AP(17), AP(18), AP(19),
                              AP(20), AP(21), AL(22), AL(23), AL(24), AL(25), AI(26), AI(27), AI(28)))

static PyObject* py_sw_set_stream(PyObject* self, PyObject* const* args, Py_ssize_t nargs) {
  (void)self;
  Arg v[1];
  if (!parse(args, nargs, "P", v, "sw_set_stream")) return NULL;
  return PyLong_FromLong(sw_set_stream(v[0].p));
}

static PyObject* py_sw_get_stream(PyObject* self, PyObject* unused) {
  (void)self;
  (void)unused;
  void* s = sw_get_stream();
  if (!s) Py_RETURN_NONE;
  return PyLong_FromVoidPtr(s);
}

static PyObject* py_sw_version(PyObject* self, PyObject* unused) {
  (void)self;
  (void)unused;
  return PyLong_FromLong(sw_version());
}

static PyObject* bytes_or_none(const char* s) {
  if (!s) Py_RETURN_NONE;
  return PyBytes_FromString(s);
}

static PyObject* py_sw_status_string(PyObject* self, PyObject* const* args, Py_ssize_t nargs) {
  (void)self;
  Arg v[1];
  if (!parse(args, nargs, "I", v, "sw_status_string")) return NULL;
  return bytes_or_none(sw_status_string(v[0].i));
}

static PyObject* py_sw_last_error(PyObject* self, PyObject* unused) {
  (void)self;
  (void)unused;
  return bytes_or_none(sw_last_error());
}

static PyObject* py_sw_last_launch(PyObject* self, PyObject* unused) {
  (void)self;
  (void)unused;
  return bytes_or_none(sw_last_launch());
}

#define FAST(NAME) {#NAME, (PyCFunction)(void (*)(void))py_##NAME, METH_FASTCALL, NULL}
#define NOARG(NAME) {#NAME, (PyCFunction)py_##NAME, METH_NOARGS, NULL}

static PyMethodDef methods[] = {
    NOARG(sw_version),
    FAST(sw_affine_scan),
    FAST(sw_affine_scan_i32),
    FAST(sw_affine_scan_noalloc),
    FAST(sw_affine_scan_schedule),
    FAST(sw_affine_scan_schedule_i32),
    FAST(sw_affine_scan_proj),
    FAST(sw_affine_scan_proj_i32),
    FAST(sw_selective_scan_fwd),
    FAST(sw_selective_scan_fwd_bf16),
    FAST(sw_selective_scan_fwd_schedule),
    FAST(sw_selective_scan_fwd_ex),
    FAST(sw_selective_scan_fwd_train),
    FAST(sw_selective_scan_bwd),
    FAST(sw_selective_scan_plan),
    FAST(sw_set_stream),
    NOARG(sw_get_stream),
    FAST(sw_status_string),
    NOARG(sw_last_error),
    NOARG(sw_last_launch),
    {NULL, NULL, 0, NULL}};

static struct PyModuleDef module = {PyModuleDef_HEAD_INIT, "_swcall",
                                    "Fast calls into libscanweaver's C ABI.", -1, methods,
                                    NULL, NULL, NULL, NULL};

PyMODINIT_FUNC PyInit__swcall(void) { return PyModule_Create(&module); }
