"""MI355X (gfx950) implementation of TCL's Mamba cost-model hot path.

  paper_2604_12891_amd.binding   ctypes binding of libtcl.so (include/tcl.h)
  paper_2604_12891_amd.workload  seeded synthetic inputs and weights
  paper_2604_12891_amd.build     hipcc build of libtcl.so

Importing the package loads nothing; the library is loaded on first use
by `binding.lib()`.
"""
