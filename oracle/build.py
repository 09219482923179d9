"""Build step for the oracle's C library (test infrastructure only)."""
from oracle.rocket_oracle import build

if __name__ == "__main__":
    print(build(force=True))
