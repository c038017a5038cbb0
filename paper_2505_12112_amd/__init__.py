"""MI355X-native incremental GNN embedding propagation (Ripple, arXiv 2505.12112).

The compute path lives in the HIP library ``libripple.so`` built from ``csrc/``;
``paper_2505_12112_amd.ripple`` is its ctypes binding and ``synth`` draws the
seeded synthetic inputs. Importing the package loads neither.
"""
__all__ = ["synth", "ripple"]
