"""Local-shard SBP linear layer on MI355X (gfx950).

The product is the C-ABI library ``libsbp.so`` (declared in ``include/sbp.h``,
built from ``csrc/``); ``sbp`` is its thin ctypes binding. Importing this
package loads nothing: ``from paper_2301_06813_amd import sbp`` loads the
library and fails loudly if it has not been built.
"""
