"""A looped LLM decode step for AMD MI355X (gfx950).

The compute path is the HIP library ``libkl.so`` built from ``csrc/``; this
package only builds it and marshals arguments to its C ABI (``binding``).
"""
