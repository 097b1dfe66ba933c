"""Multi-channel layers whose candidate plans reach every copy form of the
matrix-core kernel's private stages (each wave staging its own channels):
16-byte input copies with the staged window moved left at the map's right
edge, the 4-byte fallback where a padded row is wider than the map, 16-byte
copies of paired 32-float planes (K = 1), partial last stages in which some
waves get no channels, even K, and the 16 x 32 eight-wave shape.  Used by
tests/test_gpu_plans.py; tests/test_abi.py checks the coverage."""

PRIVATE_LAYERS = [(37, 40, 33, 20, 3), (70, 40, 28, 9, 1), (45, 48, 26, 26, 5),
                  (20, 36, 19, 21, 2), (50, 20, 10, 12, 3), (24, 40, 61, 9, 1)]
